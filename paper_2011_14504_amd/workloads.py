"""Layer shapes of the synthetic workloads (shapes only, no arithmetic).

A conv layer is (name, C_in, C_out, R, stride, pad, dilation, bn, relu).
"""

# Single 3x3 conv, stride 1, pad 1, 16 -> 16 channels on a 1x32x32 map,
# followed by L1BN over 16 channels.
SINGLE_CONV = dict(name="single-conv3x3-16", N=1, H=32, W=32, C=16,
                   layers=[("conv", 16, 16, 3, 1, 1, 1)])

# FCN-VGG16 encoder slice: conv1_1, conv1_2, maxpool 2x2/2, conv2_1, conv2_2,
# each conv followed by L1BN + ReLU; batch 8 at 224x224 (Sec. 5 crops images
# to 512x512; this slice uses the 224x224 ImageNet input of the encoder).
VGG16_BLOCKS12 = dict(name="fcn-vgg16-blocks1-2", N=8, H=224, W=224, C=3,
                      layers=[("conv", 3, 64, 3, 1, 1, 1),
                              ("conv", 64, 64, 3, 1, 1, 1),
                              ("maxpool", 2, 2, 0),
                              ("conv", 64, 128, 3, 1, 1, 1),
                              ("conv", 128, 128, 3, 1, 1, 1)])


def conv_out(H, R, stride, pad, dil):
    return (H + 2 * pad - dil * (R - 1) - 1) // stride + 1
