"""CPU oracle for the checkpointed (sublinear-memory) training step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link
or execute anything in this package: only the test-suite, the smoke check and
the benchmark's CPU-baseline leg use it.  It shares no code with the HIP path.

What it computes (Chen, Xu, Zhang, Guestrin, "Training Deep Nets with Sublinear
Memory Cost"):

* ``units``     -- forward and backward of every unit kind on the chain
                   (residual-MLP block, CIFAR stem and basic block, ImageNet stem
                   and bottleneck block, LSTM step with its softmax head) and the
                   chain heads (MSE, average-pool + FC + softmax cross-entropy),
                   in float64 by default.  bf16 storage can be emulated by
                   rounding at the points where the GPU stores bf16.
* ``nets``      -- the plain full-storage step: forward storing everything, the
                   head, then backward from the last unit to the first
                   (section 3: the explicit backward pathway in reverse
                   topological order).  This is the definition the checkpointed
                   step must reproduce exactly (section 5.1: every optimisation
                   gives an equivalent weight gradient).
* ``planner``   -- the segmentations of section 4: the sqrt(n) schedule
                   (section 4.3, Eq. 1), the budget-driven greedy segmentation
                   (Alg. 3), the recursive k=1 schedule (section 4.4, Eq. 2-3),
                   user cut lists and the single segment; with the memory
                   accounting of a static plan.
* ``schedule``  -- CPU executors of Alg. 1 (segment re-forward, then backward)
                   and of the recursive schedule, with a unit-forward counter.

Parity status of each function is stated in its module header.
"""
