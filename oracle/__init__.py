"""Plain CPU oracle of the retraining / micro-profiling / inference hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
load this package: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP library and the two
never import each other; both read inputs from the separate `synth` package.

Everything is float64 numpy in NHWC layout, written for a reader to check
against the definitions by eye:

* `rng`      - SplitMix64 and Fisher-Yates, for the uniform random training-data
               subset of micro-profiling and the per-epoch shuffle (paper,
               section 4.3, "Training data sampling").
* `nn`       - convolution, BatchNorm, ReLU, pooling, the classifier layer,
               softmax cross-entropy, SGD with momentum, bilinear resize, argmax.
* `resnet18` - the ResNet18 edge classifier (He et al., "Deep residual
               learning", the paper's reference for ResNet), torchvision topology,
               split into the stages whose freezing the paper uses as a cost
               knob (section 3.1).
* `ekya`     - retraining of the last k stages on a subsampled window with
               held-out accuracy after every epoch (sections 3.1 and 4.3),
               the micro-profiler's sweep over configurations, and inference
               at a chosen resolution (section 1, inference configurations).
"""
