"""The five workloads of the path, by their shapes (pyramid recipe, input sizes, dtype, seeds).

Plain parameters only: both the GPU path and the oracle receive them as inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field

from .synth import IMAGENET_MEAN

PAD_ZERO, PAD_RAMP = 0, 1


@dataclass(frozen=True)
class Workload:
    name: str
    H: int
    W: int
    seeds: tuple            # one image seed per image of the batch
    n_scales: int
    steps_per_octave: int
    base_scale: float = 1.0
    base_longest_side: int = 0
    pad: int = 0
    pad_mode: int = PAD_ZERO
    plane_h: int = 0        # 0 => one plane per scale
    plane_w: int = 0
    dtypes: tuple = ("f32",)
    pool5: bool = False
    n_boxes: int = 0
    box_seed: int = 0
    mean: tuple = field(default=IMAGENET_MEAN)
    aspects: tuple = ()     # aspect-ratio pyramids (empty: one pyramid)

    @property
    def n_img(self) -> int:
        return len(self.seeds)


# 227x227 image, scales 1 and 2^-0.5, no padding, each scale its own plane, fp32, pool5 on.
ALEXNET_227 = Workload("alexnet227_2scale", 227, 227, (101,), 2, 2, pad=0, dtypes=("f32",), pool5=True)
# 480x640 image, 8 scales at 2^-0.25 from longest side 1024, zero padding 16, one plane per scale.
VGA_8SCALE = Workload("vga480x640_8scale", 480, 640, (102,), 8, 4, base_longest_side=1024, pad=16,
                      pad_mode=PAD_ZERO, dtypes=("f32", "f16"))
# 768x1024 image, 25 scales at 2^-0.1, ramp padding 16, stitched onto 1200x1200 planes, fp16.
XGA_25SCALE = Workload("xga768x1024_25scale_1200plane", 768, 1024, (103,), 25, 10, pad=16,
                       pad_mode=PAD_RAMP, plane_h=1200, plane_w=1200, dtypes=("f16",))
# Batch of 16 such images, bf16.
XGA_25SCALE_B16 = Workload("xga768x1024_25scale_1200plane_batch16", 768, 1024,
                           tuple(1000 + i for i in range(16)), 25, 10, pad=16, pad_mode=PAD_RAMP,
                           plane_h=1200, plane_w=1200, dtypes=("bf16",))
# The 25-scale pyramid plus 2000 region proposals.
XGA_25SCALE_REGIONS = Workload("xga768x1024_25scale_2000regions", 768, 1024, (103,), 25, 10, pad=16,
                               pad_mode=PAD_RAMP, plane_h=1200, plane_w=1200, dtypes=("f16",),
                               n_boxes=2000, box_seed=105)

ALL = (ALEXNET_227, VGA_8SCALE, XGA_25SCALE, XGA_25SCALE_B16, XGA_25SCALE_REGIONS)
