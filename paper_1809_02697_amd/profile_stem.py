"""Workload for hardware-counter passes over ResNet-50's stem alone.

    rocprofv3 --pmc SQ_WAVES SQ_WAVE_CYCLES ... --output-format csv -d OUT -o stem -- \
        python -m paper_1809_02697_amd.profile_stem

The 3 -> 64 channel 7x7 / stride 2 / pad 3 convolution of a 224x224 image
(batch 1, NCHW16c input, BN folded, ReLU), launched 51 times through
neo_conv2d_nchwxc in one launch configuration (tile [2,1], one wave per
workgroup, no split: the tuned batch-1 choice)."""
import os

import torch

from paper_1809_02697_amd import neo, workloads as wl


def main():
    neo.lib()
    c = wl.conv_case(3, 64, 7, 7, 2, 3, 224, 224, N=1, epilogue="relu", out_hw=(112, 112))
    w, b = neo.fold_bn(c.w, c.bias, c.bn["gamma"], c.bn["beta"], c.bn["mean"], c.bn["var"],
                       c.bn["eps"])
    bias = torch.from_numpy(b).cuda()
    wp = neo.pack_filter(torch.from_numpy(w).cuda())
    x = neo.layout_transform(torch.from_numpy(c.x).cuda(), 0, 16, *c.x.shape)
    os.environ["NEO_CONV_CONFIG"] = "2,1,1,1"
    y = neo.conv2d_nchwxc(x, 3, wp, 64, 7, 7, bias=bias, stride=2, pad=3, act="relu")
    for _ in range(50):
        neo.conv2d_nchwxc(x, 3, wp, 64, 7, 7, bias=bias, stride=2, pad=3, act="relu", out=y)
    torch.cuda.synchronize()
    print("stem: 51 launches", flush=True)


if __name__ == "__main__":
    main()
