"""CPU oracle for SpecTrain's pipeline-stage step.

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, NumPy float64
statement of what one pipeline stage computes under SpecTrain weight
prediction (Chen, Yang, Cheng, "Efficient and Robust Parallel DNN Training
through Model Parallelism on Multi-GPU Platform", Section 3.2, Eq. 1-6) and of
the one-forward-one-backward pipeline order the weight versions come from
(Section 3.1). Only the tests, the smoke check and the CPU-baseline leg of the
benchmark may import it; the product library never does.

Modules:
  numerics   - storage rounding (float32 master state, bf16 operands)
  method     - Eq. 1 (smoothed gradient), the momentum weight update,
               Eq. 4 (s-step prediction), Eq. 5/6 (version differences)
  schedule   - one-forward-one-backward task order of a K-stage pipeline
  layers     - forward/backward of the layer types the stages are built from
  stages     - forward/backward of a whole stage for each workload kind
  trajectory - runs a workload for M mini-batches and records the states

Precision: arithmetic is float64. Where a workload fixes a storage precision
(float32 master W, v and g; bf16 operands and activations for bf16 stages) the
value is rounded to it at the point the stage definition stores it. Every
function states the passage it follows.

Pins (tests/test_oracle_*.py): the worked example of Section 3.2, Eq. 5 and
Eq. 6 as brute-force counts of the updates between a pass and the completion
of the round trip, a count of updates between a stage's forward and backward,
the stage-to-stage hand-off against the composed network under autograd, exact reduction to
sequential momentum SGD at s=0, the closed form under a constant gradient
with dyadic constants, gamma=1 freezing, central finite differences of every
stage kind, library special cases (torch CPU conv2d, LSTM, layer_norm,
scaled-dot-product attention, cross_entropy), and the CE value ln C at zero
logits.
"""
