"""Seeded synthetic inputs shared by the CPU oracle's tests and the HIP path.

This package holds only input generation: network definitions with seeded
random weights, and seeded synthetic video chunks whose change structure
follows the workloads described for the diff-computation experiments.
It contains none of the method's arithmetic (no convolution, masking,
thresholding or accumulation), so that the oracle and the HIP path stay
independent and only meet on identical inputs.

All arrays are NHWC float32 numpy arrays whose values are already exactly
representable in the network's storage dtype (``"f32"``, ``"f16"`` or
``"bf16"``); rounding to the dtype is done with PyTorch's own conversion.
"""

from .nets import (ACT_NONE, ACT_RELU, ACT_SILU, LayerSpec, NetSpec,
                   crnn_vgg_net, depthwise_test_net, efficientnet_mini_net,
                   efficientnet_net, resnet50_net, resnet_mini_net, toy_net,
                   to_storage)
from .video import (driving_video, object_video, multistream_video,
                    random_sparse_video, textline_video, toy_video)

__all__ = [
    "ACT_NONE", "ACT_RELU", "ACT_SILU", "LayerSpec", "NetSpec",
    "crnn_vgg_net", "depthwise_test_net", "efficientnet_mini_net",
    "efficientnet_net", "resnet50_net", "resnet_mini_net", "toy_net",
    "to_storage", "driving_video", "object_video", "multistream_video",
    "random_sparse_video", "textline_video", "toy_video",
]
