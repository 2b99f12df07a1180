"""Host-only parts of the anchor pool (no GPU): the native pool bookkeeping and the gate decision of Eq. 10-11
against the oracle, on seeded random histories and distances."""
import numpy as np
import pytest

from oracle import kvc_oracle as O
from paper_2609_34060_amd import kvc


@pytest.mark.parametrize("capacity,seed", [(3, 1), (5, 2), (6, 3), (10, 4), (20, 5)])
def test_native_pool_follows_the_oracle_rule(capacity, seed):
    rng = np.random.default_rng(seed)
    native, ref = kvc.Pool(capacity), O.AnchorPool(capacity)
    for step in range(300):
        op = rng.integers(0, 3)
        if op == 0 or step < capacity:
            length = int(rng.integers(1, 5000))
            assert native.insert(step, length) == ref.insert(step, length)
        elif op == 1:
            occupied = [i for i, e in enumerate(ref.slots) if e is not None]
            used = list(rng.choice(occupied, size=int(rng.integers(1, len(occupied) + 1))))
            native.record_use(used)
            ref.record_use(used)
        else:
            k = int(rng.integers(0, 5000))
            assert native.eligible(k) == ref.eligible(k)
    for i, e in enumerate(ref.slots):
        assert native.slot(i) == (e["id"], e["length"], e["uses"])


def test_gate_decision_matches_oracle():
    rng = np.random.default_rng(7)
    for n in range(0, 12):
        for _ in range(20):
            d = rng.uniform(0.0, 6.0, n).astype(np.float32)
            tau = float(rng.uniform(0.0, 1.0))
            acc, g, h = kvc.kvc_gate_decide(list(d), tau)
            og, oh, oacc = O.gate(d.astype(np.float64), tau)
            assert abs(h - oh) <= 1e-6 and np.allclose(g, og, atol=1e-6)
            if abs(oh - tau) > 1e-6:
                assert acc == oacc
