"""The three evaluated networks at batch 1, built once per test session
(VGG-16 alone draws 138 M parameters).  Tests must not modify them."""
import functools

from paper_1809_02697_amd import workloads as wl


@functools.lru_cache(maxsize=None)
def net(name):
    return {"resnet50": wl.resnet50, "vgg16": wl.vgg16, "inception_v3": wl.inception_v3}[name](1)


def resnet50():
    return net("resnet50")


def vgg16():
    return net("vgg16")


def inception_v3():
    return net("inception_v3")
