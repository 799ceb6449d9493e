"""The five layer configurations the sparse-sparse layer is measured on.

Each configuration is a chain of sparse-weight layers.  A layer packs N
kernels into one (complement factor n, so weight sparsity is 1 - 1/n), runs
the sparse-sparse product, optionally a 2x2 max-pool, optionally k-WTA and,
in the int8 chains, requantises the k-WTA winners back to int8.

Stand-ins (no dataset or trained weights are used):
  * config 2 has the shape of the keyword-spotting CNN of Table 1 (32x32x1
    audio features -> conv 5x5 -> pool -> conv 5x5 -> pool -> 1500 -> 12) with
    uniform int8 inputs in place of the speech data;
  * configs 3-5 have the shapes of ResNet-50 stage-1 / stage-3 layers and of a
    MobileNetV2 inverted-residual pointwise pair (Section 5) with random
    activations in place of ImageNet features.
"""
from __future__ import annotations

from dataclasses import dataclass, field

SEED_BASE = 2112_13896


@dataclass(frozen=True)
class LayerSpec:
    name: str
    kind: str                 # "conv" (NHWC input) or "linear" ([batch][d_in] input)
    c_in: int                 # conv: input channels; linear: d_in
    c_out: int                # conv: output channels; linear: d_out
    n: int                    # complement factor: kernels overlaid per packed kernel
    kh: int = 1
    kw: int = 1
    stride: int = 1
    pad: int = 0
    pool: int = 1             # 2: 2x2 stride-2 max-pool after the layer
    k: int | None = None      # k-WTA winners per row (pixel for conv); None: no k-WTA
    shift: int | None = None  # int chains: requantise winners with this shift
    bias: bool = False
    weight_dist: str = "int8"  # "int8": uniform non-zero in [-127,127]; "normal": N(0, 2/nnz_k)
    dense_input: bool = False  # the layer's input is dense: run it sparse-dense (no compaction)

    @property
    def r(self) -> int:
        """Receptive-field length (slots per kernel before packing)."""
        return self.kh * self.kw * self.c_in

    @property
    def groups(self) -> int:
        return self.c_out // self.n

    @property
    def nnz_k(self) -> int:
        """Non-zero weights per kernel."""
        return self.r // self.n


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    dtype: str                # "i8" (int8 inputs/weights, int32 sums) or "f32"
    batch: int
    in_shape: tuple           # conv nets: (H, W, C); linear: (D,)
    in_nnz: int | None        # non-zeros per input row/pixel; None = dense
    in_dist: str              # "u1_127", "u_m127_127" or "absnormal"
    layers: tuple = field(default_factory=tuple)
    description: str = ""

    @property
    def seed(self) -> int:
        return SEED_BASE + self.cid


# Requantisation shifts (int chains).  Each is the smallest s >= 0 with
# max|winner| >> s <= 127 over the seeded batch of the layer's k-WTA winners,
# computed once from the CPU reference run and frozen here; the script that derives them lives in
# tests/golden/ and a CPU test re-derives and compares them.
_C2_S1, _C2_S2, _C2_S3 = 11, 9, 9
_C5_S1 = 9

CONFIGS = {
    1: Config(
        cid=1, name="linear_i8_b16", dtype="i8", batch=16, in_shape=(512,),
        in_nnz=64, in_dist="u1_127",
        layers=(LayerSpec("linear", "linear", 512, 64, n=8, k=16, bias=True),),
        description="single linear layer 512->64, N=8, 64/512 active inputs, k-WTA 16/64",
    ),
    2: Config(
        cid=2, name="gsc_cnn_i8_b256", dtype="i8", batch=256, in_shape=(32, 32, 1),
        in_nnz=None, in_dist="u_m127_127",
        layers=(
            LayerSpec("conv1", "conv", 1, 64, n=1, kh=5, kw=5, pool=2, k=8, shift=_C2_S1,
                      dense_input=True),
            LayerSpec("conv2", "conv", 64, 64, n=16, kh=5, kw=5, pool=2, k=8, shift=_C2_S2),
            LayerSpec("linear1", "linear", 1600, 1500, n=20, k=75, shift=_C2_S3),
            LayerSpec("output", "linear", 1500, 12, n=1),
        ),
        description="keyword-spotting CNN of Table 1: conv5x5 1->64 (dense), pool, "
                    "k-WTA 8/64; conv5x5 64->64 N=16, pool, k-WTA 8/64; "
                    "linear 1600->1500 N=20, k-WTA 75/1500; dense linear 1500->12",
    ),
    3: Config(
        cid=3, name="resnet_s1_conv3x3_f32_b32", dtype="f32", batch=32, in_shape=(56, 56, 64),
        in_nnz=7, in_dist="absnormal",
        layers=(LayerSpec("conv3x3", "conv", 64, 64, n=8, kh=3, kw=3, pad=1, k=8,
                          weight_dist="normal"),),
        description="ResNet-50 stage-1 3x3 conv 64->64 at 56x56, N=8, 7/64 active, k-WTA 8/64",
    ),
    4: Config(
        cid=4, name="resnet_s3_block_f32_b64", dtype="f32", batch=64, in_shape=(14, 14, 1024),
        in_nnz=102, in_dist="absnormal",
        layers=(
            LayerSpec("conv1x1", "conv", 1024, 256, n=16, k=26, weight_dist="normal"),
            LayerSpec("conv3x3", "conv", 256, 256, n=16, kh=3, kw=3, pad=1, k=26,
                      weight_dist="normal"),
        ),
        description="ResNet-50 stage-3 1x1 1024->256 then 3x3 256->256 at 14x14, N=16, "
                    "10% active, k-WTA 26/256 after each",
    ),
    5: Config(
        cid=5, name="mbv2_pointwise_i8_b128", dtype="i8", batch=128, in_shape=(14, 14, 96),
        in_nnz=12, in_dist="u1_127",
        layers=(
            LayerSpec("expand", "conv", 96, 576, n=8, k=72, shift=_C5_S1, bias=True),
            LayerSpec("project", "conv", 576, 96, n=8, bias=True),
        ),
        description="MobileNetV2 pointwise pair 1x1 96->576 (N=8, k-WTA 72/576) then "
                    "1x1 576->96 (N=8), 12/96 active inputs",
    ),
}


def get_config(cid: int) -> Config:
    return CONFIGS[int(cid)]
