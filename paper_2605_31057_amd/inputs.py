"""Seeded synthetic inputs and workload shapes.

Holds no part of the method's arithmetic: only shapes, mask parameters and
a seeded draw of Q, K, V.  Both the library's tests/bench and the oracle are
fed from here.

Recipe: one CPU ``torch.Generator`` seeded with 16 (the paper's seed) draws,
for each head in turn, Q then K then V as float32 N(0, 1) of shape [N, 128];
an optional factor scales the values; values are rounded to bfloat16
(round to nearest even) and laid out [heads, N, 128] contiguous.  Drawing per
head keeps the first heads of a workload identical whatever the head count.
"""
from dataclasses import dataclass, field

D = 128


@dataclass(frozen=True)
class Workload:
    name: str
    heads: int
    frames: int           # T, latent frames
    tokens_per_frame: int  # P = latent height x width
    block: int
    budget_frames: int    # C
    window: int           # W
    tper: int = 0         # 0: derived from C and W
    steps: tuple = (10,)  # denoising steps the mask is built for
    layers: tuple = (0,)
    value_scale: float = 1.0
    text_tokens: int = 0   # text tokens after the video tokens (dual-stream)
    desc: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def n_tokens(self):
        return self.frames * self.tokens_per_frame + self.text_tokens

    @property
    def n_blocks(self):
        return -(-self.n_tokens // self.block)


WORKLOADS = {
    # 1 head, 4 latent frames of 16x16, block 64; a one-frame window (W = 0)
    # and one rotating anchor (T_per = 4).
    "tiny": Workload("tiny", 1, 4, 256, 64, budget_frames=2, window=0, tper=4,
                     steps=(0, 1, 2, 3),
                     desc="1 head, 4 x 16x16 tokens, block 64, W=0, T_per=4"),
    # Same shape, W = 1: every frame attends to all 4 frames (full mask).
    "tiny_full": Workload("tiny_full", 1, 4, 256, 64, budget_frames=4, window=1,
                          tper=4, steps=(0,),
                          desc="tiny shape with a full mask (W=1, T_per=4)"),
    # Wan 2.1 1.3B self-attention at the 81-frame training horizon:
    # 21 latent frames of 30x52, 12 heads; values scaled by 1/sqrt(128).
    "wan13_1x": Workload("wan13_1x", 12, 21, 1560, 128, budget_frames=21, window=6,
                         steps=(10,), value_scale=128 ** -0.5,
                         desc="Wan2.1-1.3B layer, 21 x 30x52 tokens, 12 heads"),
    # Wan 2.1 1.3B at a 6x horizon (481 frames -> 121 latent frames).
    "wan13_6x": Workload("wan13_6x", 12, 121, 1560, 128, budget_frames=21, window=6,
                         steps=tuple(range(50)),
                         desc="Wan2.1-1.3B layer, 121 x 30x52 tokens, 12 heads"),
    # Wan 2.1 14B at the 6x horizon: 40 heads.
    "wan14_6x": Workload("wan14_6x", 40, 121, 1560, 128, budget_frames=21, window=6,
                         steps=(10,),
                         desc="Wan2.1-14B layer, 121 x 30x52 tokens, 40 heads"),
    # HunyuanVideo 1.5 (480p) at a 2x horizon (257 frames -> 65 latent
    # frames of 30x53), 16 heads; C = 33 from a 129-frame training horizon.
    "hv15_2x": Workload("hv15_2x", 16, 65, 1590, 128, budget_frames=33, window=6,
                        steps=tuple(range(50)), layers=(0, 1, 2, 3),
                        desc="HunyuanVideo-1.5 layer, 65 x 30x53 tokens, 16 heads"),
    # The same layer with the Wan budget C = 21 instead of 33 (a labelled
    # variant: C = 33 leaves 30 of 33 frames at the 1x horizon).
    "hv15_2x_c21": Workload("hv15_2x_c21", 16, 65, 1590, 128, budget_frames=21, window=6,
                            steps=(0, 10),
                            desc="HunyuanVideo-1.5 layer, 65 x 30x53 tokens, 16 heads, C=21"),
    # The same layer with the dual-stream text tokens in self-attention: 512
    # text tokens (prompts of about 500 tokens) after the video tokens.
    "hv15_2x_text": Workload("hv15_2x_text", 16, 65, 1590, 128, budget_frames=33,
                             window=6, steps=(0, 10), text_tokens=512,
                             desc="HunyuanVideo-1.5 layer, 65 x 30x53 video + 512 "
                                  "text tokens, 16 heads"),
}


def make_qkv(heads, n_tokens, seed=16, value_scale=1.0, d=D):
    """(q, k, v) bfloat16 CPU tensors [heads, n_tokens, d] from the recipe."""
    import torch
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    out = [torch.empty((heads, n_tokens, d), dtype=torch.bfloat16) for _ in range(3)]
    for h in range(heads):
        for t in out:
            x = torch.randn((n_tokens, d), generator=g, dtype=torch.float32)
            if value_scale != 1.0:
                x.mul_(value_scale)
            t[h].copy_(x.to(torch.bfloat16))
    return tuple(out)


def workload_qkv(w, heads=None, seed=16):
    """Inputs of workload ``w`` (optionally only its first ``heads`` heads)."""
    return make_qkv(heads or w.heads, w.n_tokens, seed=seed, value_scale=w.value_scale)
