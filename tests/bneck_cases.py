"""Bottleneck-ResNet parity cases shared by the CPU conditioning checks and
the GPU tests, and the conditioning measure both use.

Conditioning.  With a batch norm after every bf16-rounded convolution the
network is chaotic at the rounding level: a value whose accumulation lands on
the other side of a bf16 rounding midpoint moves its channel's statistics,
which moves the channel and flips further roundings downstream, and where a
ReLU input crosses zero a gradient term of full size appears or vanishes.
Multiplying every value by (1 + 1e-7 N(0, 1)) just before it is rounded to
bf16 -- the size of the fp32 accumulation error of these small sums --
measures how far such flips move each gradient tensor.  WELL_POSED shapes are
those where six such perturbed oracle runs stay within 2e-3 (max-abs
relative) of the unperturbed run on every tensor; on them the GPU must match
the bf16-emulating oracle to a fixed bar.  CHAOTIC shapes (more blocks,
batch 1-4, real stage widths) move by up to tens of percent under the same
perturbation, so there only what no rounding can change is compared: plans
against each other bit for bit, the peak bytes and the forward counts.  The
single operators at real widths are pinned separately (test_gpu_ops_bf16).
"""
import numpy as np

JITTER, REPS, GATE = 1e-7, 6, 2e-3

_B = dict(kind="resnet_bottleneck", expansion=4)

WELL_POSED = {
    # stem + a stride-1 projection block
    "p1": dict(_B, stage_blocks=(1,), widths=(16,), stem_channels=16, image=16, batch=2, classes=7,
               seed=91),
    # + a stride-2 projection block
    "p11": dict(_B, stage_blocks=(1, 1), widths=(8, 16), stem_channels=8, image=16, batch=2,
                classes=7, seed=104),
    # projection block + identity block
    "p2": dict(_B, stage_blocks=(2,), widths=(8,), stem_channels=8, image=16, batch=2, classes=7,
               seed=111),
    # projection + identity + stride-2 projection
    "p21": dict(_B, stage_blocks=(2, 1), widths=(8, 16), stem_channels=16, image=16, batch=2,
                classes=7, seed=127),
}

CHAOTIC = {
    "b22": dict(_B, stage_blocks=(2, 2), widths=(8, 16), stem_channels=8, image=16, batch=2, classes=7,
                seed=91),
    # four stages down to 1 x 1
    "b2111": dict(_B, stage_blocks=(2, 1, 1, 1), widths=(8, 16, 32, 64), stem_channels=16, image=32,
                  batch=2, classes=10, seed=91),
    # expansion 2, a single image
    "b121": dict(_B, stage_blocks=(1, 2, 1), widths=(8, 16, 32), expansion=2, stem_channels=8,
                 image=32, batch=1, classes=5, seed=92),
    # the real stage-1/2 channel counts: several GEMM tiles, split-K weight gradients
    "wide": dict(_B, stage_blocks=(1, 1), widths=(64, 128), stem_channels=64, image=64, batch=4,
                 classes=100, seed=83),
}


def maxrel(g, o):
    g = np.asarray(g, np.float64).reshape(-1)
    o = np.asarray(o, np.float64).reshape(-1)
    return float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-30))


def oracle_runs(d):
    """The float64 bf16-emulating oracle, the plain float64 oracle, and per
    tensor the largest deviation of six perturbed emulating runs."""
    from oracle import nets, units as U
    chain = lambda prec: nets.Chain(d["structure"], d["params"], prec)
    le, ge = nets.full_storage_step(chain(U.Prec(np.float64, True)), d["input"], d["target"])
    lf, gf = nets.full_storage_step(chain(U.Prec(np.float64, False)), d["input"], d["target"])
    env = {k: 0.0 for k in ge}
    lenv = 0.0
    for s in range(REPS):
        prec = U.Prec(np.float64, True, JITTER, np.random.default_rng(700 + s))
        lj, gj = nets.full_storage_step(chain(prec), d["input"], d["target"])
        lenv = max(lenv, abs(lj - le) / abs(le))
        for k in ge:
            env[k] = max(env[k], maxrel(gj[k], ge[k]))
    return (le, ge), (lf, gf), env, lenv
