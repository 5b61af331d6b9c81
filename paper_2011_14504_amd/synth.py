"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke
check.  This module holds no arithmetic of the method: it only draws random
numbers (numpy PCG64) with the shapes and value ranges of the workloads.

Recipe (stands in for PASCAL VOC 2012 / ADE20K, which are not available):
  * images, activations: int8 codes uniform on [-127, 127], exponent -7;
  * errors arriving at a layer output: int8 codes uniform on [-127, 127],
    exponent -20 (values up to ~1.2e-4, the 1e-5..1e-4 range the paper
    reports for errors in Sec. 3.1.2);
  * conv weights: float32 He-normal N(0, 2/fan_in) (MSRA initialisation,
    Sec. 3.2.1), turned into 24-bit master codes by the library's own Eq. 7
    quantizer on each side;
  * BN gamma/beta: gamma = 1, beta = 0 for benchmark runs; random int8 codes
    for parity runs;
  * labels: uint8 uniform over the class count.
Seeds: 1450400 + 100 * workload + ordinal.
"""
import numpy as np

SEED_BASE = 1450400
ACT_EXP = -7
ERR_EXP = -20


def seed_for(workload, ordinal):
    return SEED_BASE + 100 * int(workload) + int(ordinal)


def rng(seed):
    return np.random.Generator(np.random.PCG64(int(seed)))


def int_codes(seed, shape, lo=-127, hi=127, dtype=np.int8):
    """Integers uniform on [lo, hi]."""
    return rng(seed).integers(lo, hi + 1, size=shape, dtype=np.int64).astype(dtype)


def he_normal(seed, shape, fan_in):
    """float32 normal with standard deviation sqrt(2 / fan_in)."""
    std = np.sqrt(2.0 / float(fan_in))
    return (rng(seed).standard_normal(size=shape) * std).astype(np.float32)


def bilinear_filter(R, cin, cout):
    """The bilinear-upsampling initialisation of a transposed conv (the FCN
    decoder, Sec. 3.2.1): w[c][r][s][c] = f(r) f(s) on the channel diagonal,
    f(t) = 1 - |t - centre| / factor with factor = ceil(R / 2) and centre =
    factor - 1 (R odd) or factor - 1/2 (R even); zero off the diagonal.
    Layout [cin][R][R][cout]; float32 (every value is a multiple of
    1/factor^2, exact)."""
    factor = (R + 1) // 2
    centre = factor - 1 if R % 2 == 1 else factor - 0.5
    f = 1.0 - np.abs(np.arange(R) - centre) / factor
    w = np.zeros((cin, R, R, cout), dtype=np.float32)
    for c in range(min(cin, cout)):
        w[c, :, :, c] = np.outer(f, f)
    return w


def gaussian_codes(seed, shape, std, dtype=np.int8):
    """Rounded normal samples clipped to [-127, 127] (for BN statistics tests)."""
    v = np.rint(rng(seed).standard_normal(size=shape) * std)
    return np.clip(v, -127, 127).astype(dtype)


def labels(seed, shape, classes):
    return rng(seed).integers(0, classes, size=shape, dtype=np.int64).astype(np.uint8)


def uniform_f32(seed, shape, lo=-1.0, hi=1.0):
    return rng(seed).uniform(lo, hi, size=shape).astype(np.float32)


# ---------------------------------------------------------------------------
# workload shapes (shapes and seeds only)
# ---------------------------------------------------------------------------
# A workload is a list of nodes in topological order; each node names its
# input node(s) ("input" is the workload's input tensor):
#   conv     src, cin, cout, R, stride, pad, dil, bn, relu
#            conv -> SQ8; then, if bn, L1BN (+ ReLU if relu) -> Q_A
#   maxpool  src, k, stride, pad
#   add      srcs = [a, b], relu: residual merge SQ8(ReLU(a + b))
#   gap      src: global average pooling over H x W -> [N,1,1,C]
#   concat   srcs: channel concatenation, SQ8; a [N,1,1,C] source (the
#            image-pooling branch) is broadcast over the spatial size first
# The last node is the output.  loss = "given": an int8 error (uniform codes,
# exponent -20) arrives at the output; "softmax_ce": the output logits are
# upsampled bilinearly to the image size and scored against per-pixel labels.


def conv(name, src, cin, cout, R, stride=1, pad=0, dil=1, bn=True, relu=True):
    return dict(kind="conv", name=name, src=[src], cin=cin, cout=cout, R=R, stride=stride,
                pad=pad, dil=dil, bn=bn, relu=relu)


def deconv(name, src, cin, cout, R, stride, pad, relu=False):
    """Transposed convolution (a decoder's learned upsampling): the adjoint
    of a conv whose input is this node's output ([N, (H-1) stride - 2 pad +
    R, ..., cout]) and whose output is this node's input; its weights are
    that conv's, [cin][R][R][cout].  No BN (the FCN decoder has none)."""
    return dict(kind="conv", transposed=True, name=name, src=[src], cin=cin, cout=cout, R=R,
                stride=stride, pad=pad, dil=1, bn=False, relu=relu)


def maxpool(name, src, k, stride, pad=0):
    return dict(kind="maxpool", name=name, src=[src], k=k, stride=stride, pad=pad)


def add_relu(name, a, b):
    return dict(kind="add", name=name, src=[a, b], relu=True)


def add(name, a, b):
    """Sum of two maps without a ReLU (the FCN's score fusion)."""
    return dict(kind="add", name=name, src=[a, b], relu=False)


def gap(name, src):
    return dict(kind="gap", name=name, src=[src])


def concat(name, srcs):
    return dict(kind="concat", name=name, src=list(srcs))


def bottleneck(prefix, src, cin, mid, cout, stride=1, dil=1, proj=False):
    """ResNet-50 v1.5 bottleneck: 1x1 -> 3x3 (stride, dilation) -> 1x1 (L1BN,
    no ReLU), projection shortcut (1x1 with the stride, L1BN, no ReLU) when
    the shape changes, ReLU after the residual add."""
    nodes = []
    sc = src
    if proj:
        nodes.append(conv(prefix + ".proj", src, cin, cout, 1, stride, 0, 1, relu=False))
        sc = prefix + ".proj"
    nodes.append(conv(prefix + ".conv1", src, cin, mid, 1))
    nodes.append(conv(prefix + ".conv2", prefix + ".conv1", mid, mid, 3, stride, dil, dil))
    nodes.append(conv(prefix + ".conv3", prefix + ".conv2", mid, cout, 1, relu=False))
    nodes.append(add_relu(prefix + ".out", prefix + ".conv3", sc))
    return nodes, prefix + ".out"


def res_stage(prefix, src, cin, mid, cout, blocks, stride=1, dil_first=1, dil_rest=1):
    nodes = []
    for b in range(blocks):
        nb, src = bottleneck(f"{prefix}.{b}", src, cin if b == 0 else cout, mid, cout,
                             stride if b == 0 else 1, dil_first if b == 0 else dil_rest,
                             proj=(b == 0))
        nodes += nb
    return nodes, src


def aspp(prefix, src, cin, classes, rates=(6, 12, 18), mid=256):
    """DeepLabv3 ASPP head: 1x1 branch, three 3x3 atrous branches (pad =
    dilation), image pooling (GAP -> 1x1 -> L1BN + ReLU, broadcast back),
    concatenation, 1x1 fuse, 1x1 classifier (no BN, no ReLU)."""
    nodes = [conv(prefix + ".b0", src, cin, mid, 1)]
    for i, d in enumerate(rates):
        nodes.append(conv(f"{prefix}.b{i + 1}", src, cin, mid, 3, 1, d, d))
    nodes.append(gap(prefix + ".pool", src))
    nodes.append(conv(prefix + ".b4", prefix + ".pool", cin, mid, 1))
    nodes.append(concat(prefix + ".cat", [f"{prefix}.b{i}" for i in range(5)]))
    nodes.append(conv(prefix + ".fuse", prefix + ".cat", 5 * mid, mid, 1))
    nodes.append(conv(prefix + ".cls", prefix + ".fuse", mid, classes, 1, bn=False, relu=False))
    return nodes, prefix + ".cls"


def resnet50_os16(src="input"):
    """ResNet-50 v1.5 backbone at output stride 16: layer4 keeps stride 1 and
    uses dilation 2 in its blocks 1-2 (block 0 keeps dilation 1)."""
    nodes = [conv("stem", src, 3, 64, 7, 2, 3),
             maxpool("pool", "stem", 3, 2, 1)]
    out = "pool"
    for name, mid, cout, blocks, stride, d0, d1 in (("layer1", 64, 256, 3, 1, 1, 1),
                                                    ("layer2", 128, 512, 4, 2, 1, 1),
                                                    ("layer3", 256, 1024, 6, 2, 1, 1),
                                                    ("layer4", 512, 2048, 3, 1, 1, 2)):
        cin = 64 if name == "layer1" else mid * 2
        nb, out = res_stage(name, out, cin, mid, cout, blocks, stride, d0, d1)
        nodes += nb
    return nodes, out


# Single 3x3 conv 16 -> 16, stride 1, pad 1, on a 1x32x32 map, then L1BN over
# 16 channels; the input gradient is computed too.
SINGLE_CONV = dict(id=1, name="single-conv3x3-16ch-32x32-n1", N=1, H=32, W=32, C=16,
                   input_grad=True, loss="given",
                   nodes=[conv("conv", "input", 16, 16, 3, 1, 1)])

# FCN-VGG16 encoder slice: conv1_1, conv1_2, maxpool 2x2/2, conv2_1, conv2_2,
# batch 8 of 3x224x224 images; no gradient is taken w.r.t. the image.
VGG16_BLOCKS12 = dict(id=2, name="fcn-vgg16-blocks1-2-n8-224", N=8, H=224, W=224, C=3,
                      input_grad=False, loss="given",
                      nodes=[conv("conv1_1", "input", 3, 64, 3, 1, 1),
                             conv("conv1_2", "conv1_1", 64, 64, 3, 1, 1),
                             maxpool("pool1", "conv1_2", 2, 2, 0),
                             conv("conv2_1", "pool1", 64, 128, 3, 1, 1),
                             conv("conv2_2", "conv2_1", 128, 128, 3, 1, 1)])

# ResNet-50 stage conv2_x: three bottlenecks 64 -> (64, 64, 256), the first
# with a projection shortcut, on batch 16 of 64x56x56 features.
RESNET50_CONV2X = dict(id=3, name="resnet50-conv2x-n16-56", N=16, H=56, W=56, C=64,
                       input_grad=True, loss="given",
                       nodes=res_stage("conv2_x", "input", 64, 64, 256, 3)[0])

# DeepLabv3 ASPP head on batch 8 of 2048x32x32 features, 21 classes.
ASPP_HEAD = dict(id=4, name="deeplabv3-aspp-2048ch-32x32-n8", N=8, H=32, W=32, C=2048,
                 input_grad=True, loss="given",
                 nodes=aspp("aspp", "input", 2048, 21)[0])

# Full DeepLabv3-ResNet50 training step at output stride 16: batch 8 of
# 3x512x512 images, 150 classes (ADE20K's count), per-pixel labels.
_R50 = resnet50_os16()
DEEPLABV3_R50 = dict(id=5, name="deeplabv3-r50-os16-n8-512", N=8, H=512, W=512, C=3,
                     input_grad=False, loss="softmax_ce", classes=150,
                     nodes=_R50[0] + aspp("aspp", _R50[1], 2048, 150)[0])



def fcn8s(classes, src="input"):
    """FCN8s on VGG16 (no BN): the five conv blocks with max pooling, the
    fully convolutional fc6 (7x7, 4096) and fc7 (1x1, 4096) with ReLU, the
    score convs (1x1, no ReLU) on fc7, pool4 and pool3, and three transposed
    convs initialised as bilinear upsampling (x2, x2, x8) with the score
    fusions between them.  Padding is chosen so that each upsampling
    doubles (or multiplies by 8) the map exactly, so no crop is needed."""
    nodes, prev, cin = [], src, 3
    for b, (c, n) in enumerate([(64, 2), (128, 2), (256, 3), (512, 3), (512, 3)], 1):
        for i in range(1, n + 1):
            nodes.append(conv(f"conv{b}_{i}", prev, cin, c, 3, 1, 1, bn=False))
            prev, cin = f"conv{b}_{i}", c
        nodes.append(maxpool(f"pool{b}", prev, 2, 2, 0))
        prev = f"pool{b}"
    nodes += [conv("fc6", "pool5", 512, 4096, 7, 1, 3, bn=False),
              conv("fc7", "fc6", 4096, 4096, 1, bn=False),
              conv("score_fr", "fc7", 4096, classes, 1, bn=False, relu=False),
              deconv("upscore2", "score_fr", classes, classes, 4, 2, 1),
              conv("score_pool4", "pool4", 512, classes, 1, bn=False, relu=False),
              add("fuse_pool4", "upscore2", "score_pool4"),
              deconv("upscore_pool4", "fuse_pool4", classes, classes, 4, 2, 1),
              conv("score_pool3", "pool3", 256, classes, 1, bn=False, relu=False),
              add("fuse_pool3", "upscore_pool4", "score_pool3"),
              deconv("upscore8", "fuse_pool3", classes, classes, 16, 8, 4)]
    return nodes


# FCN8s-VGG16 training step: batch 8 of 3x512x512 images, 21 classes (PASCAL
# VOC), MSE loss against the one-hot labels, gradients by Eq. 18 (no BN).
FCN8S_VGG16 = dict(id=6, name="fcn8s-vgg16-n8-512", N=8, H=512, W=512, C=3, input_grad=False,
                   loss="mse", classes=21, gq=2, nodes=fcn8s(21))

WORKLOADS = {1: SINGLE_CONV, 2: VGG16_BLOCKS12, 3: RESNET50_CONV2X, 4: ASPP_HEAD,
             5: DEEPLABV3_R50, 6: FCN8S_VGG16}


def without_bn(wl):
    """The same graph with every conv's L1BN removed (the paper's FCN has no
    BN); a conv's ReLU then follows its output quantizer's input."""
    d = dict(wl)
    d["name"] = wl["name"] + "-nobn"
    d["nodes"] = [dict(n, bn=False) if n["kind"] == "conv" else n for n in wl["nodes"]]
    return d


def scaled(wl, N=None, H=None, W=None):
    """The same workload at another batch or input size (parity tests)."""
    d = dict(wl)
    if N is not None:
        d["N"] = N
    if H is not None:
        d["H"] = H
    if W is not None:
        d["W"] = W
    return d


def node_shapes(wl):
    """Output shape [N, H, W, C] of every node (pure shape arithmetic)."""
    shapes = {"input": (wl["N"], wl["H"], wl["W"], wl["C"])}
    for nd in wl["nodes"]:
        N, H, W, Cc = shapes[nd["src"][0]]
        k = nd["kind"]
        if k == "conv" and nd.get("transposed"):
            P = (H - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
            Q = (W - 1) * nd["stride"] - 2 * nd["pad"] + nd["dil"] * (nd["R"] - 1) + 1
            shapes[nd["name"]] = (N, P, Q, nd["cout"])
        elif k == "conv":
            P = (H + 2 * nd["pad"] - nd["dil"] * (nd["R"] - 1) - 1) // nd["stride"] + 1
            Q = (W + 2 * nd["pad"] - nd["dil"] * (nd["R"] - 1) - 1) // nd["stride"] + 1
            shapes[nd["name"]] = (N, P, Q, nd["cout"])
        elif k == "maxpool":
            shapes[nd["name"]] = (N, (H + 2 * nd["pad"] - nd["k"]) // nd["stride"] + 1,
                                  (W + 2 * nd["pad"] - nd["k"]) // nd["stride"] + 1, Cc)
        elif k == "add":
            shapes[nd["name"]] = (N, H, W, Cc)
        elif k == "gap":
            shapes[nd["name"]] = (N, 1, 1, Cc)
        elif k == "concat":
            sp = [shapes[s] for s in nd["src"]]
            Hs = max(t[1] for t in sp)
            Ws = max(t[2] for t in sp)
            shapes[nd["name"]] = (N, Hs, Ws, sum(t[3] for t in sp))
        else:
            raise ValueError(k)
    return shapes


def conv_nodes(wl):
    return [nd for nd in wl["nodes"] if nd["kind"] == "conv"]


def workload_inputs(wl, N=None):
    """Seeded inputs of a workload: image/activation codes, float weights per
    conv (He-normal), and either the error arriving at the output or the
    per-pixel labels."""
    wl = scaled(wl, N)
    N = wl["N"]
    x = int_codes(seed_for(wl["id"], 0), (N, wl["H"], wl["W"], wl["C"]))
    weights = []
    for i, nd in enumerate(conv_nodes(wl)):
        R, cin, cout = nd["R"], nd["cin"], nd["cout"]
        if nd.get("transposed"):
            weights.append(bilinear_filter(R, cin, cout))
        else:
            weights.append(he_normal(seed_for(wl["id"], i + 1), (cout, R, R, cin), cin * R * R))
    out = dict(x=x, x_exp=ACT_EXP, weights=weights, seed=seed_for(wl["id"], 0))
    shp = node_shapes(wl)[wl["nodes"][-1]["name"]]
    if wl["loss"] == "given":
        out["dy"] = int_codes(seed_for(wl["id"], 50), shp)
        out["dy_exp"] = ERR_EXP
    else:
        out["labels"] = labels(seed_for(wl["id"], 51), (N, wl["H"], wl["W"]), wl["classes"])
    if wl["loss"] == "mse":
        out["labels"] = labels(seed_for(wl["id"], 51), shp[:3], wl["classes"])
    return out
