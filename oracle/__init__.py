"""CPU oracle for the Adaptive SGD hot path (arXiv 2110.07029).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The product path (the
HIP library and its Python binding) never calls it and shares no code with it.

Plain, slow, obviously correct NumPy in float64 (float32 storage for the model
parameters, which is what the method trains):

* ``model``   - the 3-layer sparse MLP of Sec. 5.1 ("Datasets and Model"):
                CSR input -> W1 -> ReLU -> W2 -> softmax + cross-entropy, its
                gradient and the SGD update (Sec. 2.1, "Stochastic Gradient
                Descent"), prediction and the init generator.
* ``elastic`` - batch-size scaling (Alg. 1), normalized merge weights and the
                momentum merge (Alg. 2), and the dynamic mega-batch dispatch
                (Sec. 3.1) replayed from a schedule.

Every function is pinned by tests under ``tests/`` against values the paper or
mathematics fixes (finite differences, closed forms, dense equivalents, the
worked batch-scaling case of Sec. 3.1, published splitmix64 outputs).
"""
