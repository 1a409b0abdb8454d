"""The device step state's table (lt_step_table, host only) against the oracle's step
scalars: for every t in 1..20000 and 3000 sampled t up to 10^6, fp32(lr / (1 -
beta1^t)) from the table's fp64 entry (the device's fp64 division, emulated here by
numpy's IEEE division and fp32 rounding) and the table's rbc2 equal lto_step_scalars
bitwise, for several learning rates and betas (App. C hyperparameters and others)."""
import numpy as np

import oracle
import paper_2608_11919_amd as lt


def test_step_table_gives_the_oracles_scalars():
    rng = np.random.default_rng(5)
    configs = ((1e-4, 0.9, 0.999), (1e-5, 0.9, 0.999), (3e-3, 0.5, 0.9999), (0.1, 0.0, 0.0),
               (2.5e-4, 0.99, 0.95))
    for lr, b1, b2 in configs:
        dense = lt.lt_step_table(b1, b2, 1, 20000)
        sampled = sorted(int(t) for t in rng.integers(20001, 10**6 + 1, size=3000))
        ts = list(range(1, 20001)) + sampled
        entries = list(dense) + [lt.lt_step_table(b1, b2, t, 1)[0] for t in sampled]
        for t, e in zip(ts, entries):
            o = oracle.step_scalars(lr, b1, b2, 1e-8, 0.01, t)
            size = np.float32(np.float64(lr) / np.float64(e["one_minus_beta1_t"]))
            assert size.tobytes() == o["step_size"].tobytes(), (lr, b1, b2, t)
            assert np.float32(e["rbc2"]).tobytes() == o["rbc2"].tobytes(), (lr, b1, b2, t)


def test_step_table_arguments():
    L = lt.lib()
    assert lt.lt_step_state_bytes(0) == 0 and lt.lt_step_state_bytes(4) == 64 + 4 * 16
    assert L.lt_step_table(1.0, 0.9, 1, 1, None) == lt.LT_ERR_INVALID_ARG
    assert L.lt_step_table(0.9, 0.9, 0, 1, None) == lt.LT_ERR_INVALID_ARG
    assert L.lt_step_table(0.9, 0.9, 1, 0, None) == lt.LT_OK
