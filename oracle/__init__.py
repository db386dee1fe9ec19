"""Plain CPU oracle for the LSTM-PPO optimizer step of OpenAI Five (arXiv:1912.06680).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package smoke check and the
CPU-baseline leg of the benchmark may import this package.  The product path
(the HIP library and its Python binding) never imports, links or calls it, and
this package imports nothing from the product.

Every function is a direct, slow, fp64 NumPy statement of what the paper's
method computes, written so that it can be checked against the paper by eye:

* ``lstm``   -- single-layer forget-gate LSTM forward and truncated
                backpropagation through time (section "Training System",
                subsections "Playing Dota using AI" and "Optimizing the Policy").
* ``gae``    -- generalized advantage estimation over rollout segments
                (subsection "Optimizing the Policy"; Table "Hyperparameters").
* ``ppo``    -- linear policy/value heads, PPO clipped surrogate, value loss
                and entropy bonus, with gradients (subsection "Optimizing the
                Policy"; appendix "Exploration", subsection "Loss function";
                appendix "Neural Network Architecture").
* ``prelstm`` -- the LSTM's input side: running observation normalisation,
                the pre-LSTM fully-connected layer and the cross-hero
                max-pool, forward and backward (appendices "Observation
                Space" and "Neural Network Architecture").
* ``surgery`` -- widening the LSTM and extending its input on the flat
                parameter vector, with Adam's moments (appendix "Surgery").
* ``reward`` -- reward post-processing ahead of GAE: game time weighting,
                team spirit, zero sum, normalisation by a running standard
                deviation (appendix "Reward Weights"; Table "Hyperparameters").
* ``adam``   -- Adam with the per-parameter gradient clip to +-5 sqrt(v)
                (subsection "Optimizing the Policy"; Table "Hyperparameters").
* ``philox`` -- Philox4x64-10 counter-based generator and Gumbel-max action
                sampling (sampling an action each timestep, subsection
                "Playing Dota using AI").
* ``bf16``   -- round-to-nearest-even fp32 -> bfloat16, used to build the
                bf16-path reference inputs.
* ``step``   -- the composition of the above into one optimizer step.

Pinning: every function is checked in ``tests/test_oracle_*.py`` against values
the mathematics fixes (finite differences, closed forms, brute force,
invariants) or against an independent library routine (PyTorch CPU float64
LSTMCell / autograd / Adam / Categorical, NumPy's Philox bit generator).
"""
