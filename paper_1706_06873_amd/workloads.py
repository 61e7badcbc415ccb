"""Seeded synthetic convolution layers shaped like the paper's CNN workloads.

This module only draws inputs: it holds none of the convolution's arithmetic
and is shared by the tests, the benchmark and the smoke check. Every tensor is
drawn on the CPU from a ``torch.Generator`` seeded with the layer's seed: the
unpadded input interior first, then the kernel; the interior is then placed
inside a ring of zeros (the paper assumes padding is already applied to the
input, Section 2.1). bf16 layers are drawn in fp32 and rounded to bf16 with
round-to-nearest-even.

Layouts follow Table 1 of the paper: I is i_n x i_h x i_w x i_c, K is
k_h x k_w x i_c x k_c.
"""
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Layer:
    name: str
    i_n: int
    ih_int: int      # unpadded input height
    iw_int: int      # unpadded input width
    i_c: int
    k_h: int
    k_w: int
    k_c: int
    s_h: int
    s_w: int
    pad: int         # zero ring added around the interior
    dtype: str       # "f32" or "bf16": element type of I and K
    i_dist: str      # "u11" (uniform[-1,1]), "u01" (uniform[0,1])
    k_dist: str      # "u11", "n0.1", "n0.01" (normal, mean 0, that std)
    seed: int
    note: str = ""

    @property
    def i_h(self):
        return self.ih_int + 2 * self.pad

    @property
    def i_w(self):
        return self.iw_int + 2 * self.pad

    @property
    def dims(self):
        """(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w) in the paper's notation."""
        return (self.i_n, self.i_h, self.i_w, self.i_c, self.k_h, self.k_w, self.k_c,
                self.s_h, self.s_w)


# The five layers: sizes, value distributions and seeds.
LAYERS = {
    "tiny": Layer("tiny", 1, 7, 7, 1, 3, 3, 1, 1, 1, 0, "f32", "u11", "u11", 0,
                  "7x7 input, 3x3 kernel, the size of the example of Figs. 1 and 2"),
    "resnet_mid": Layer("resnet_mid", 32, 56, 56, 64, 3, 3, 64, 1, 1, 1, "f32", "u11", "u11", 1,
                        "ResNet-style 56x56x64 mid layer (Table 2, cv9 shape, padded to 58)"),
    "vgg_first": Layer("vgg_first", 16, 224, 224, 3, 3, 3, 64, 1, 1, 1, "f32", "u01", "n0.1", 2,
                       "VGG-style first layer (Table 2, cv7 shape, padded to 226)"),
    "alexnet_conv1": Layer("alexnet_conv1", 128, 227, 227, 3, 11, 11, 96, 4, 4, 0, "f32", "u01",
                           "n0.01", 3, "AlexNet conv1, 11x11 stride 4 (Table 2, cv1)"),
    "deep_bf16": Layer("deep_bf16", 256, 14, 14, 512, 3, 3, 512, 1, 1, 1, "bf16", "u11", "u11", 4,
                       "deep narrow-spatial 14x14x512 layer, bf16 inputs (cv11/cv12-like)"),
}
LAYER_ORDER = ["tiny", "resnet_mid", "vgg_first", "alexnet_conv1", "deep_bf16"]

# The twelve benchmark layers of Table 2 (input i_h x i_w x i_c, kernel
# k_h x k_w x k_c, stride), taken as printed: no padding is added.
TABLE2 = {
    "cv1": (227, 227, 3, 11, 11, 96, 4),
    "cv2": (231, 231, 3, 11, 11, 96, 4),
    "cv3": (227, 227, 3, 7, 7, 64, 2),
    "cv4": (224, 224, 64, 7, 7, 64, 2),
    "cv5": (24, 24, 96, 5, 5, 256, 1),
    "cv6": (12, 12, 256, 3, 3, 512, 1),
    "cv7": (224, 224, 3, 3, 3, 64, 1),
    "cv8": (112, 112, 64, 3, 3, 128, 1),
    "cv9": (56, 56, 64, 3, 3, 64, 1),
    "cv10": (28, 28, 128, 3, 3, 128, 1),
    "cv11": (14, 14, 256, 3, 3, 256, 1),
    "cv12": (7, 7, 512, 3, 3, 512, 1),
}

# Table 3 weighs five Table 2 layers by how often ResNet-101 uses them.
TABLE3_WEIGHTS = {"cv4": 1, "cv9": 3, "cv10": 4, "cv11": 23, "cv12": 3}


def table2_layer(name, i_n=32, dtype="f32", stride=None, dist="u11"):
    """A Table 2 layer at batch i_n; ``stride`` overrides s_h = s_w (the
    stride sweep of Fig. 4(a) runs cv1 with s = 1..10). Seed: the layer's
    number (cv1 -> 101, ..., cv12 -> 112), plus 100 * stride when overridden."""
    i_h, i_w, i_c, k_h, k_w, k_c, s = TABLE2[name]
    num = int(name[2:])
    seed = 100 + num + (100 * stride if stride else 0)
    s = stride or s
    return Layer("%s%s" % (name, "_s%d" % stride if stride else ""), i_n, i_h, i_w, i_c, k_h, k_w,
                 k_c, s, s, 0, dtype, dist, dist, seed,
                 "Table 2 %s: %dx%dx%d input, %dx%dx%d kernel, stride %d"
                 % (name, i_h, i_w, i_c, k_h, k_w, k_c, s))


def _draw(gen, shape, dist):
    if dist == "u11":
        return torch.rand(shape, generator=gen, dtype=torch.float32) * 2.0 - 1.0
    if dist == "u01":
        return torch.rand(shape, generator=gen, dtype=torch.float32)
    if dist.startswith("n"):
        std = float(dist[1:])
        return torch.randn(shape, generator=gen, dtype=torch.float32) * std
    if dist == "int":  # small integers in [-3, 3]: every partial sum stays exact in fp32
        return torch.randint(-3, 4, shape, generator=gen).to(torch.float32)
    raise ValueError("unknown distribution %r" % dist)


def make_inputs(layer: Layer, i_n: int = None, round_bf16: bool = True):
    """Draw (I, K) for a layer on the CPU. ``i_n`` overrides the batch size
    (the first i_n images of the full draw are NOT reproduced; a smaller batch
    is a separate draw with the same seed). With ``round_bf16=False`` a bf16
    layer is returned as the fp32 values before rounding."""
    n = layer.i_n if i_n is None else i_n
    gen = torch.Generator(device="cpu")
    gen.manual_seed(layer.seed)
    interior = _draw(gen, (n, layer.ih_int, layer.iw_int, layer.i_c), layer.i_dist)
    K = _draw(gen, (layer.k_h, layer.k_w, layer.i_c, layer.k_c), layer.k_dist)
    p = layer.pad
    if p:
        I = torch.zeros((n, layer.i_h, layer.i_w, layer.i_c), dtype=torch.float32)
        I[:, p:p + layer.ih_int, p:p + layer.iw_int, :] = interior
    else:
        I = interior.contiguous()
    if layer.dtype == "bf16" and round_bf16:
        I = I.to(torch.bfloat16)
        K = K.to(torch.bfloat16)
    return I.contiguous(), K.contiguous()


def random_case(seed, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype="f32", dist="u11"):
    """Seeded random (I, K) of arbitrary shape for parity sweeps (no padding)."""
    layer = Layer("case%d" % seed, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, 0, dtype,
                  dist, dist, seed)
    return make_inputs(layer)


def to_oracle_array(t):
    """CPU tensor -> numpy array in the oracle's convention (bf16 as uint16 bits)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError("unsupported dtype %s" % t.dtype)
