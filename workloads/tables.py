"""Per-layer segment tables for the five gradient workloads.

Each trainable layer contributes a weight segment then a bias segment, in
layer order.  A fully-connected layer is the 1x1-filter special case of a
convolution (Sec. 3 "Preliminaries").  Weight counts follow Eq. 1 without its
byte factor: channels * filters * filter width * filter height.

Layout rule: every segment starts on a multiple of ALIGN elements (256 B of
fp32, 128 B of fp16), the gap before it is zero padding that belongs to no
segment and is never read into a sum nor written.

This module describes workload shapes only; it holds none of the method's
arithmetic and is shared by the oracle-side tests and the GPU benchmark.
"""
from dataclasses import dataclass, field
from typing import List, Tuple

ALIGN = 64


@dataclass(frozen=True)
class Layer:
    name: str
    out_ch: int
    in_ch: int      # input channels seen by one filter (after grouping)
    kh: int = 1
    kw: int = 1

    @property
    def weights(self):
        return self.out_ch * self.in_ch * self.kh * self.kw

    @property
    def fan_in(self):
        return self.in_ch * self.kh * self.kw


@dataclass(frozen=True)
class Segment:
    name: str
    offset: int
    length: int
    fan_in: int
    is_bias: bool
    layer: Layer
    lr_mult: float = 1.0
    decay_mult: float = 1.0


@dataclass
class Workload:
    """A synthetic gradient-aggregation workload (K workers, one segment
    table) with the solver settings of the network it imitates."""
    name: str
    layers: List[Layer]
    K: int
    dtype: str                      # replica storage: "f32" or "f16"
    batch: int
    lr: float
    mu: float
    wd: float
    grad_std: str                   # "fan_in" -> 1e-3/sqrt(fan_in), else a number as text
    weight_init: str                # "gauss0.01", "nin", "xavier_bias0.2"
    segments: List[Segment] = field(default_factory=list)
    padded: int = 0                 # one past the last padded element (multiple of ALIGN)

    @property
    def n_params(self):
        return sum(s.length for s in self.segments)

    @property
    def s_g(self):
        return 2 if self.dtype == "f16" else 4

    def table(self, lr_mults=None):
        """(offset, length, lr_mult, decay_mult) rows, in segment order."""
        return [(s.offset, s.length, s.lr_mult, s.decay_mult) for s in self.segments]

    def algorithmic_bytes(self, out=False, bcast=False):
        """Bytes one fused step must move: K replicas read, w and v read,
        w' and v' written; +4N for the raw sum, +4NK for the broadcast."""
        n = self.n_params
        b = n * (self.K * self.s_g + 16)
        if out:
            b += 4 * n
        if bcast:
            b += 4 * n * self.K
        return b


def _round_up(x, a):
    return (x + a - 1) // a * a


def lay_out(layers, bias=True, caffe_bias_mults=False):
    """Weight then bias segment per layer, each start aligned to ALIGN."""
    segs, off = [], 0
    for L in layers:
        parts = [(L.name + ".w", L.weights, False)]
        if bias:
            parts.append((L.name + ".b", L.out_ch, True))
        for nm, n, isb in parts:
            off = _round_up(off, ALIGN)
            lm, dm = ((2.0, 0.0) if (isb and caffe_bias_mults) else (1.0, 1.0))
            segs.append(Segment(nm, off, n, L.fan_in, isb, L, lm, dm))
            off += n
    return segs, _round_up(off, ALIGN)


def conv(name, o, i, k=1):
    return Layer(name, o, i, k, k)


def nin_layers():
    return [conv("conv1", 96, 3, 11), conv("cccp1", 96, 96), conv("cccp2", 96, 96),
            conv("conv2", 256, 96, 5), conv("cccp3", 256, 256), conv("cccp4", 256, 256),
            conv("conv3", 384, 256, 3), conv("cccp5", 384, 384), conv("cccp6", 384, 384),
            conv("conv4", 1024, 384, 3), conv("cccp7", 1024, 1024), conv("cccp8", 1000, 1024)]


# Inception modules of GoogLeNet v1: (name, c_in, #1x1, #3x3red, #3x3, #5x5red, #5x5, #pool_proj)
INCEPTION = [("3a", 192, 64, 96, 128, 16, 32, 32), ("3b", 256, 128, 128, 192, 32, 96, 64),
             ("4a", 480, 192, 96, 208, 16, 48, 64), ("4b", 512, 160, 112, 224, 24, 64, 64),
             ("4c", 512, 128, 128, 256, 24, 64, 64), ("4d", 512, 112, 144, 288, 32, 64, 64),
             ("4e", 528, 256, 160, 320, 32, 128, 128), ("5a", 832, 256, 160, 320, 32, 128, 128),
             ("5b", 832, 384, 192, 384, 48, 128, 128)]


def googlenet_layers(aux=False):
    L = [conv("conv1/7x7_s2", 64, 3, 7), conv("conv2/3x3_reduce", 64, 64, 1),
         conv("conv2/3x3", 192, 64, 3)]
    for nm, cin, n1, r3, n3, r5, n5, pp in INCEPTION:
        p = f"inception_{nm}/"
        L += [conv(p + "1x1", n1, cin), conv(p + "3x3_reduce", r3, cin), conv(p + "3x3", n3, r3, 3),
              conv(p + "5x5_reduce", r5, cin), conv(p + "5x5", n5, r5, 5), conv(p + "pool_proj", pp, cin)]
        if aux and nm in ("4a", "4d"):
            tag = "loss1" if nm == "4a" else "loss2"
            cin_aux = 512 if nm == "4a" else 528
            L += [conv(f"{tag}/conv", 128, cin_aux), conv(f"{tag}/fc", 1024, 2048),
                  conv(f"{tag}/classifier", 1000, 1024)]
    L.append(conv("loss3/classifier", 1000, 1024))
    return L


def vgg19_layers():
    chans = [(64, 3), (64, 64), (128, 64), (128, 128), (256, 128), (256, 256), (256, 256), (256, 256),
             (512, 256), (512, 512), (512, 512), (512, 512), (512, 512), (512, 512), (512, 512), (512, 512)]
    L = [conv(f"conv{i + 1}", o, c, 3) for i, (o, c) in enumerate(chans)]
    L += [conv("fc6", 4096, 25088), conv("fc7", 4096, 4096), conv("fc8", 1000, 4096)]
    return L


def alexnet_layers(grouped=True):
    g = 2 if grouped else 1
    return [conv("conv1", 96, 3, 11), conv("conv2", 256, 96 // g, 5), conv("conv3", 384, 256, 3),
            conv("conv4", 384, 384 // g, 3), conv("conv5", 256, 384 // g, 3),
            conv("fc6", 4096, 9216), conv("fc7", 4096, 4096), conv("fc8", 1000, 4096)]


def _make(name, layers, caffe_bias_mults=False, **kw):
    wl = Workload(name=name, layers=layers, **kw)
    wl.segments, wl.padded = lay_out(layers, caffe_bias_mults=caffe_bias_mults)
    return wl


def flat():
    """One flat fp32 segment of 2^20 elements, K=4."""
    wl = Workload(name="flat", layers=[Layer("flat", 1 << 20, 1)], K=4, dtype="f32", batch=256,
                  lr=0.01, mu=0.9, wd=5e-4, grad_std="1e-3", weight_init="gauss0.01")
    L = wl.layers[0]
    wl.segments = [Segment("flat", 0, 1 << 20, 1, False, L)]
    wl.padded = 1 << 20
    return wl


def nin():
    """Network-in-Network (ImageNet) shapes, K=32 fp32; solver of Sec. 7.1 item 2."""
    return _make("nin", nin_layers(), K=32, dtype="f32", batch=256, lr=0.01, mu=0.9, wd=5e-4,
                 grad_std="fan_in", weight_init="nin")


def googlenet(aux=False, caffe_bias=False):
    """GoogLeNet v1 shapes (57 convolutions + FC), K=128 fp32, batch 1024,
    lr 0.08 (Sec. 7.3 "Ultra-deep models"), mu 0.9, wd 2e-4 (Sec. 7.1).
    caffe_bias: every bias segment takes twice the learning rate and no
    weight decay (lr_mult 2, decay_mult 0), as in the Caffe network
    definitions the paper trains with (Sec. 7.1 item 2)."""
    name = "googlenet" + ("_aux" if aux else "") + ("_caffe_bias" if caffe_bias else "")
    return _make(name, googlenet_layers(aux), caffe_bias_mults=caffe_bias, K=128, dtype="f32",
                 batch=1024, lr=0.08, mu=0.9, wd=2e-4, grad_std="fan_in", weight_init="xavier_bias0.2")


def vgg19():
    """VGG-19 shapes, K=16 fp32, gradients N(0, 1e-4)."""
    return _make("vgg19", vgg19_layers(), K=16, dtype="f32", batch=256, lr=0.01, mu=0.9, wd=5e-4,
                 grad_std="1e-4", weight_init="gauss0.01")


def alexnet(grouped=True):
    """AlexNet shapes (grouped conv2/4/5 as released with Caffe), K=128,
    fp16 replicas with fp32 accumulation, weights and velocity."""
    return _make("alexnet" + ("" if grouped else "_ungrouped"), alexnet_layers(grouped), K=128,
                 dtype="f16", batch=256, lr=0.01, mu=0.9, wd=5e-4, grad_std="fan_in",
                 weight_init="gauss0.01")


WORKLOADS = {"flat": flat, "nin": nin, "googlenet": googlenet, "vgg19": vgg19, "alexnet": alexnet}


VARIANTS = ("googlenet_aux", "googlenet_caffe_bias", "alexnet_ungrouped")


def get(name):
    if name == "googlenet_aux":
        return googlenet(aux=True)
    if name == "googlenet_caffe_bias":
        return googlenet(caffe_bias=True)
    if name == "alexnet_ungrouped":
        return alexnet(grouped=False)
    return WORKLOADS[name]()


def eq1_weight_bytes(layers) -> int:
    """Eq. 1: bytes of all conv + FC weights in fp32 (biases not counted)."""
    return sum(L.weights * 4 for L in layers)


def segment_rows(segs) -> List[Tuple[int, int, float, float]]:
    return [(s.offset, s.length, s.lr_mult, s.decay_mult) for s in segs]
