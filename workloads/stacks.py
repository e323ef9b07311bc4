"""The five synthetic layer stacks, written out layer by layer.

Every layer lists its input spatial size explicitly, so nothing here computes
a convolution or pooling output shape; the path under test and the oracle each
derive output shapes on their own and the tests check them against the next
layer's listed input size.

Tensors are named slots: "x" is the stack input, "y" the stack output, any
other name is an intermediate tensor.

Stacks (batch, input):
  0  single layer   b1,  1x28x28x64 2-bit codes, 3x3 s1 p1 64->64
  1  AlexNet body   b32, 27x27x96 codes: conv2 5x5 96->256, pool 3/2,
                    conv3-5 3x3 at 13x13, pool5 3/2 (first and last layers of
                    the network are full precision and not part of the body)
  2  VGG-16 convs   b16, 224x224x64 codes (conv1_2 .. conv5_3, five 2x2/2 pools)
  3  ResNet-18 body b64, 56x56x64 codes: eight basic blocks, three 1x1/2
                    downsample convs with int32 output, residual joins
  4  Tiny-YOLOv2    b8, 416x416x3 8-bit codes: c1..c8 with six pools (the
                    sixth is 2x2 stride 1 "same"), 1x1 head with int32 output
"""
from dataclasses import dataclass, field
from typing import Optional, Tuple, List


@dataclass(frozen=True)
class Conv:
    name: str
    src: str
    dst: str
    h: int          # input height
    w: int          # input width
    cin: int
    cout: int
    k: int          # square kernel
    stride: int
    pad: int
    in_bits: int    # bits per input code (2, or 8 for a first layer on raw pixels)
    out_bits: int   # bits per output code; 0 means the int32 sum is the output
    # residual join: None, ("identity", slot) or ("conv", slot, down_layer_name)
    join: Optional[Tuple] = None


@dataclass(frozen=True)
class Pool:
    name: str
    src: str
    dst: str
    h: int
    w: int
    c: int
    k: int
    stride: int
    mode: str       # "valid" or "same" (window clipped at the bottom/right edge)
    bits: int = 2


def _c(name, src, dst, hw, cin, cout, k, s, p, inb=2, outb=2, join=None):
    return Conv(name, src, dst, hw, hw, cin, cout, k, s, p, inb, outb, join)


def _p(name, src, dst, hw, c, k, s, mode="valid", bits=2):
    return Pool(name, src, dst, hw, hw, c, k, s, mode, bits)


def _config0():
    return [_c("conv", "x", "y", 28, 64, 64, 3, 1, 1)]


def _config1():
    return [
        _c("conv2", "x", "t0", 27, 96, 256, 5, 1, 2),
        _p("pool2", "t0", "t1", 27, 256, 3, 2),
        _c("conv3", "t1", "t2", 13, 256, 384, 3, 1, 1),
        _c("conv4", "t2", "t3", 13, 384, 384, 3, 1, 1),
        _c("conv5", "t3", "t4", 13, 384, 256, 3, 1, 1),
        _p("pool5", "t4", "y", 13, 256, 3, 2),
    ]


def _config2():
    L = []
    a, b = "t0", "t1"
    def nxt():
        nonlocal a, b
        a, b = b, a
    # conv1_2 reads the stack input
    L.append(_c("conv1_2", "x", a, 224, 64, 64, 3, 1, 1))
    L.append(_p("pool1", a, b, 224, 64, 2, 2)); nxt()
    L.append(_c("conv2_1", a, b, 112, 64, 128, 3, 1, 1)); nxt()
    L.append(_c("conv2_2", a, b, 112, 128, 128, 3, 1, 1)); nxt()
    L.append(_p("pool2", a, b, 112, 128, 2, 2)); nxt()
    L.append(_c("conv3_1", a, b, 56, 128, 256, 3, 1, 1)); nxt()
    L.append(_c("conv3_2", a, b, 56, 256, 256, 3, 1, 1)); nxt()
    L.append(_c("conv3_3", a, b, 56, 256, 256, 3, 1, 1)); nxt()
    L.append(_p("pool3", a, b, 56, 256, 2, 2)); nxt()
    L.append(_c("conv4_1", a, b, 28, 256, 512, 3, 1, 1)); nxt()
    L.append(_c("conv4_2", a, b, 28, 512, 512, 3, 1, 1)); nxt()
    L.append(_c("conv4_3", a, b, 28, 512, 512, 3, 1, 1)); nxt()
    L.append(_p("pool4", a, b, 28, 512, 2, 2)); nxt()
    L.append(_c("conv5_1", a, b, 14, 512, 512, 3, 1, 1)); nxt()
    L.append(_c("conv5_2", a, b, 14, 512, 512, 3, 1, 1)); nxt()
    L.append(_c("conv5_3", a, b, 14, 512, 512, 3, 1, 1)); nxt()
    L.append(_p("pool5", a, "y", 14, 512, 2, 2))
    return L


def _config3():
    L = []
    cur = "x"
    n_tmp = [0]

    def tmp():
        n_tmp[0] += 1
        return "t%d" % n_tmp[0]

    stages = [(1, 64, 56), (2, 128, 56), (3, 256, 28), (4, 512, 14)]
    cin = 64
    for si, cout, hw_in in stages:
        for bi in range(2):
            pre = "l%d.%d" % (si, bi)
            downsample = (bi == 0 and si > 1)
            s1 = 2 if downsample else 1
            hw1 = hw_in if bi == 0 else hw_in // (2 if si > 1 else 1)
            hw_out = hw1 // s1
            mid = tmp()
            L.append(_c(pre + ".conv1", cur, mid, hw1, cin, cout, 3, s1, 1))
            if downsample:
                dn = tmp()
                L.append(_c(pre + ".down", cur, dn, hw1, cin, cout, 1, 2, 0,
                            outb=0))
                join = ("conv", dn, pre + ".down")
            else:
                join = ("identity", cur)
            last = (si == 4 and bi == 1)
            out = "y" if last else tmp()
            L.append(_c(pre + ".conv2", mid, out, hw_out, cout, cout, 3, 1, 1,
                        join=join))
            cur = out
            cin = cout
    return L


def _config4():
    L = []
    L.append(_c("c1", "x", "a1", 416, 3, 16, 3, 1, 1, inb=8))
    L.append(_p("p1", "a1", "b1", 416, 16, 2, 2))
    L.append(_c("c2", "b1", "a2", 208, 16, 32, 3, 1, 1))
    L.append(_p("p2", "a2", "b2", 208, 32, 2, 2))
    L.append(_c("c3", "b2", "a3", 104, 32, 64, 3, 1, 1))
    L.append(_p("p3", "a3", "b3", 104, 64, 2, 2))
    L.append(_c("c4", "b3", "a4", 52, 64, 128, 3, 1, 1))
    L.append(_p("p4", "a4", "b4", 52, 128, 2, 2))
    L.append(_c("c5", "b4", "a5", 26, 128, 256, 3, 1, 1))
    L.append(_p("p5", "a5", "b5", 26, 256, 2, 2))
    L.append(_c("c6", "b5", "a6", 13, 256, 512, 3, 1, 1))
    L.append(_p("p6", "a6", "b6", 13, 512, 2, 1, mode="same"))
    L.append(_c("c7", "b6", "a7", 13, 512, 512, 3, 1, 1))
    L.append(_c("c8", "a7", "a8", 13, 512, 512, 3, 1, 1))
    L.append(_c("head", "a8", "y", 13, 512, 30, 1, 1, 0, outb=0))
    return L


@dataclass(frozen=True)
class StackConfig:
    index: int
    name: str
    batch: int
    layers: Tuple
    in_bits: int
    description: str


CONFIGS = {
    0: StackConfig(0, "single_conv_b1", 1, tuple(_config0()), 2,
                   "single 3x3 s1 p1 conv, 64->64 at 28x28, batch 1"),
    1: StackConfig(1, "alexnet_body_b32", 32, tuple(_config1()), 2,
                   "AlexNet-shaped quantized body, batch 32"),
    2: StackConfig(2, "vgg16_convs_b16", 16, tuple(_config2()), 2,
                   "VGG-16-shaped quantized convs, batch 16, 224x224"),
    3: StackConfig(3, "resnet18_body_b64", 64, tuple(_config3()), 2,
                   "ResNet-18-shaped quantized stack, batch 64, 224x224"),
    4: StackConfig(4, "tiny_yolov2_b8", 8, tuple(_config4()), 8,
                   "Tiny-YOLOv2-shaped face-detector stack, batch 8, 416x416"),
}


def get_stack(index):
    return CONFIGS[index]


def stack_names():
    return {k: v.name for k, v in CONFIGS.items()}
