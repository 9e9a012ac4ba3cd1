"""Seeded synthetic inputs and the layer shapes of the benchmark workloads.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no arithmetic of the pruning method: only shapes, seeds and the random
draws that stand in for trained weights and real feature maps.

The paper evaluates on ILSVRC-2012 with pre-trained MobileNet and ResNet-50
weights (Sec. 4.1); neither is available here.  Stand-ins:

* weights  - He-normal, std = sqrt(2 / (Cin * kh * kw)) (fan-in);
* activations - ReLU(N(0, 1)) (ReLU6 for the MobileNet-V2 shapes), as a
  post-activation feature map.

Generation: ``torch.Generator('cpu').manual_seed(seed)``; per layer the weight
is drawn first, then the input, both in float32.  bf16 values come from the
float32 draw by round-to-nearest-even (``Tensor.to(torch.bfloat16)``).
"""
from .configs import (ConvLayer, Workload, all_workloads, config0, config1, config2, config3, nhwc,
                      config4, fc_resnet50, mobilenet_v2_pointwise, resnet50_convs)
from .gen import gen_activation, gen_integer_layer, gen_layer, gen_weight
from .sampling import sample_outputs

__all__ = ["ConvLayer", "Workload", "all_workloads", "config0", "config1", "config2", "config3", "nhwc",
           "config4", "fc_resnet50", "mobilenet_v2_pointwise", "resnet50_convs", "gen_activation",
           "gen_integer_layer", "gen_layer", "gen_weight", "sample_outputs"]
