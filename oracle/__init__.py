"""CPU oracle for the Caffe convolution layer, its pooling/LRN glue, the
softmax loss and the SGD update.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP library (``paper_1408_5093_amd``) and never touches a GPU.
"""
from .ref import (  # noqa: F401
    conv_out_shape,
    conv_forward,
    conv_backward,
    maxpool_forward,
    maxpool_backward,
    lrn_forward,
    lrn_backward,
    num_threads,
)
from .solver import learning_rate, sgd_step, softmax_loss  # noqa: F401
