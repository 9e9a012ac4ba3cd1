"""Layer shapes of the five synthetic workloads (shapes only, no arithmetic).

The networks are the ones the paper prunes (Sec. 4.1): ResNet-50 and
MobileNet-V2 at 224x224 input.  Their trained weights and ImageNet inputs are
not used; see the package docstring for the stand-ins.
"""
from dataclasses import dataclass, field, replace
from typing import List, Tuple


@dataclass(frozen=True)
class ConvLayer:
    name: str
    cin: int
    cout: int
    k: int           # square kernel kh = kw = k
    stride: int
    pad: int
    H: int           # input height = width
    N: int           # 1xN block length
    p: float         # pruning rate
    rearrange: bool  # output-channel rearrangement by filter l1 norm (Sec. 3.3)
    seed: int
    act: str = "relu"  # "relu" or "relu6" stand-in activation

    @property
    def Ho(self) -> int:
        return (self.H + 2 * self.pad - self.k) // self.stride + 1

    def out_pixels(self, batch: int) -> int:
        return batch * self.Ho * self.Ho


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    dtype: str                    # "f32" or "bf16" for X and W
    out_dtype: str                # "f32" or "bf16" for Y
    layers: Tuple[ConvLayer, ...] = field(default_factory=tuple)
    description: str = ""
    fc_layout: str = ""           # "rows" / "cols" for a fully connected layer, "" for convs
    layout: str = "nchw"          # activation layout of the convs: "nchw" or "nhwc"


def config0() -> Workload:
    """3x3/s1/p1 conv, B=1, 64->64, 56x56, fp32, N=4, p=0.5, seed 0."""
    layer = ConvLayer("conv3x3_64_64_56", 64, 64, 3, 1, 1, 56, N=4, p=0.5, rearrange=False, seed=0)
    return Workload("conv3x3_b1_64x64_56_n4_p50_f32", 1, "f32", "f32", (layer,),
                    "single 3x3 conv, stride 1, pad 1, batch 1, 64->64, 56x56, fp32, N=4, p=0.5")


def config1() -> Workload:
    """1x1 conv, B=32, 256->512, 28x28, fp32, N=16, p=0.5, rearranged."""
    layer = ConvLayer("conv1x1_256_512_28", 256, 512, 1, 1, 0, 28, N=16, p=0.5, rearrange=True,
                      seed=1000)
    return Workload("conv1x1_b32_256x512_28_n16_p50_rearranged_f32", 32, "f32", "f32", (layer,),
                    "1x1 pointwise conv, batch 32, 256->512, 28x28, fp32, N=16, p=0.5, "
                    "output-channel rearrangement")


def resnet50_convs(N: int = 32, p: float = 0.5, seed_base: int = 2000) -> List[ConvLayer]:
    """All 53 convolutions of ResNet-50 (v1.5: stride on the 3x3), 224x224 input.

    The 7x7/2 stem is dense (p = 0); the 52 bottleneck and downsample convs are
    1xN-pruned at rate p.  The stem output passes a 3x3/2 max-pool (56x56)."""
    layers = [ConvLayer("stem7x7", 3, 64, 7, 2, 3, 224, N=N, p=0.0, rearrange=False,
                        seed=seed_base)]
    cin, H = 64, 56
    idx = 1
    for stage, (blocks, width) in enumerate(zip([3, 4, 6, 3], [64, 128, 256, 512])):
        cout = width * 4
        for b in range(blocks):
            stride = 2 if (b == 0 and stage > 0) else 1
            pre = f"s{stage + 1}b{b + 1}"
            layers.append(ConvLayer(f"{pre}_1x1a", cin, width, 1, 1, 0, H, N, p, False,
                                    seed_base + idx)); idx += 1
            layers.append(ConvLayer(f"{pre}_3x3", width, width, 3, stride, 1, H, N, p, False,
                                    seed_base + idx)); idx += 1
            Ho = (H + 2 - 3) // stride + 1
            layers.append(ConvLayer(f"{pre}_1x1b", width, cout, 1, 1, 0, Ho, N, p, False,
                                    seed_base + idx)); idx += 1
            if b == 0:
                layers.append(ConvLayer(f"{pre}_down", cin, cout, 1, stride, 0, H, N, p, False,
                                        seed_base + idx)); idx += 1
            cin, H = cout, Ho
    return layers


def config2() -> Workload:
    return Workload("resnet50_b64_n32_p50_f32", 64, "f32", "f32", tuple(resnet50_convs()),
                    "all convolutions of a ResNet-50-shaped network, 224x224, batch 64, fp32, "
                    "N=32, p=0.5 per layer, stem dense")


def mobilenet_v2_pointwise(N: int, p: float, seed_base: int = 3000) -> List[ConvLayer]:
    """The 33 pointwise (1x1) convs of MobileNet-V2 (width 1.0, 224x224):
    16 expand + 17 project.  Depthwise convs, stem and head are not included."""
    settings = [(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1),
                (6, 160, 3, 2), (6, 320, 1, 1)]
    layers = []
    cin, H = 32, 112
    idx = 0
    for t, c, nrep, s in settings:
        for i in range(nrep):
            stride = s if i == 0 else 1
            hidden = cin * t
            pre = f"c{c}_{i + 1}"
            if t != 1:
                layers.append(ConvLayer(f"{pre}_expand", cin, hidden, 1, 1, 0, H, N, p, False,
                                        seed_base + idx, act="relu6")); idx += 1
            Ho = (H + 2 - 3) // stride + 1       # the depthwise 3x3 carries the stride
            layers.append(ConvLayer(f"{pre}_project", hidden, c, 1, 1, 0, Ho, N, p, False,
                                    seed_base + idx, act="relu6")); idx += 1
            cin, H = c, Ho
    return layers


def config3(N: int = 16, p: float = 0.5) -> Workload:
    return Workload(f"mobilenetv2_pw_b128_n{N}_p{int(round(p * 100))}_f32", 128, "f32", "f32",
                    tuple(mobilenet_v2_pointwise(N, p)),
                    f"MobileNet-V2 pointwise expand/project convs, batch 128, fp32, N={N}, p={p}")


def config4(out_dtype: str = "bf16") -> Workload:
    layer = ConvLayer("conv1x1_2048_2048_14", 2048, 2048, 1, 1, 0, 14, N=32, p=0.7,
                      rearrange=False, seed=4000)
    return Workload(f"conv1x1_b256_2048x2048_14_n32_p70_bf16_out{out_dtype}", 256, "bf16",
                    out_dtype, (layer,),
                    "1x1 conv, batch 256, 2048->2048, 14x14, bf16 X and W, fp32 accumulation, "
                    "N=32, p=0.7")


def fc_resnet50(N: int = 32, layout: str = "rows") -> Workload:
    """The classifier of ResNet-50 as a 1xN-pruned FC layer (Sec. 3.1: the
    kh = kw = 1 case): 2048 -> 1000 at batch 256, fp32, p = 0.5.  1000 is not
    a multiple of 32, so at N = 32 the last col-group is ragged.  `layout`:
    "rows" ([batch][2048]) or "cols" ([2048][batch])."""
    layer = ConvLayer("fc_2048_1000", 2048, 1000, 1, 1, 0, 1, N=N, p=0.5, rearrange=False,
                      seed=5000 + N)
    return Workload(f"fc_b256_2048x1000_n{N}_p50_f32_{layout}", 256, "f32", "f32", (layer,),
                    f"ResNet-50 classifier as an FC layer, batch 256, 2048->1000, fp32, N={N}, "
                    f"p=0.5, input [{'batch][2048' if layout == 'rows' else '2048][batch'}]",
                    fc_layout=layout)


def nhwc(wl: Workload) -> Workload:
    """The same workload with NHWC activations ([batch][H][W][channels] in and
    out): the gather of Eq. 8 then picks single values out of each pixel's row
    of channels."""
    return replace(wl, name=wl.name + "_nhwc", layout="nhwc",
                   description=wl.description + ", NHWC activations")


def all_workloads() -> List[Workload]:
    out = [config0(), config1(), config2()]
    for N in (4, 8, 16, 32):
        for p in (0.3, 0.5, 0.7):
            out.append(config3(N, p))
    out += [config4("bf16"), config4("f32")]
    out += [fc_resnet50(N, lay) for N in (4, 32) for lay in ("rows", "cols")]
    out += [nhwc(config1()), nhwc(config3(16, 0.5)), nhwc(config3(32, 0.5))]
    return out
