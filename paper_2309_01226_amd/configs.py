"""Named model configurations (plain values only, no arithmetic of the method).

The workloads mirror the paper's fine-tuning tasks (Saturn, arXiv 2309.01226,
Table 3 and Sec. 5 "Workloads": GPT-2 and GPT-J on text, ViT on images) at the
shapes of their public architectures:

  tiny   2-layer GPT-2-style decoder, d 64, 4 heads, MLP 256, vocab 512, seq 32, batch 2
  gpt2s  GPT-2-small shape: 12 layers, d 768, 12 heads, MLP 3072, vocab 50257, seq 1024, batch 8
  gptj   GPT-J-6B shape: 28 layers, d 4096, 16 heads (dh 256, rotary on 64), parallel
         attention+MLP block, MLP 16384, vocab 50400, seq 2048, batch 2
  vith   ViT-Huge/14 shape: 32 layers, d 1280, 16 heads, MLP 5120, 224x224x3 images,
         14x14 patches (256 + CLS = 257 tokens), 1000 classes, batch 64
  gpt2m  GPT-2-medium shape (one member of the model-selection grid): 24 layers, d 1024,
         16 heads, MLP 4096, vocab 50257, seq 512; batch, lr and frozen k vary per member
  resnet the paper's 200 M-parameter ResNet: bottleneck ResNet of ResNet-152 depth
         (3, 8, 36, 3 blocks) at twice the standard width (stem 128), 224x224x3 images,
         1000 classes, batch 64, lr 1e-4 (236 M parameters)
"""

PRESETS = {
    "tiny": dict(arch="gpt2", n_layers=2, d_model=64, n_heads=4, d_mlp=256, vocab=512,
                 seq_len=32, batch=2, lr=1e-3),
    "gpt2s": dict(arch="gpt2", n_layers=12, d_model=768, n_heads=12, d_mlp=3072, vocab=50257,
                  seq_len=1024, batch=8, lr=6e-5),
    "gptj": dict(arch="gptj", n_layers=28, d_model=4096, n_heads=16, d_mlp=16384, vocab=50400,
                 seq_len=2048, batch=2, rotary_dim=64, lr=1e-5),
    "vith": dict(arch="vit", n_layers=32, d_model=1280, n_heads=16, d_mlp=5120, vocab=1000,
                 img_size=224, patch=14, channels=3, batch=64, lr=1e-5),
    "gpt2m": dict(arch="gpt2", n_layers=24, d_model=1024, n_heads=16, d_mlp=4096, vocab=50257,
                  seq_len=512, batch=8, lr=1e-5),
    "resnet": dict(arch="resnet", n_layers=50, res_blocks=(3, 8, 36, 3), res_width=128, vocab=1000,
                   img_size=224, channels=3, batch=64, lr=1e-4),
}

# Model-selection grid: lr x batch, each member freezing k in {0, 12}; k = 12
# exactly when (lr index + batch index) is odd, so every lr and every batch
# size meets both k values.
GRID_LRS = (1e-5, 3e-5, 1e-4, 3e-4)
GRID_BATCHES = (8, 16)


def grid_members():
    out = []
    for i, lr in enumerate(GRID_LRS):
        for j, b in enumerate(GRID_BATCHES):
            c = dict(PRESETS["gpt2m"])
            c.update(lr=lr, batch=b, frozen_layers=12 if (i + j) % 2 else 0)
            out.append(c)
    return out


def preset(name, **over):
    c = dict(PRESETS[name])
    c.update(over)
    return c
