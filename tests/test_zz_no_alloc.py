"""lionmuon_step_noalloc (static device scratch, no allocation) against
lionmuon_step_ex on the same inputs, through the C ABI.

Both entry points run the same kernels on the same plan, so their results
must agree bitwise; each step is also checked against the fp64 oracle.
Consecutive calls change the list (the second is smaller), the step kind and
the tensor addresses, so the scratch's tables and address table are
rewritten between calls.
"""
import numpy as np
import pytest
import torch

from paper_2605_19811_amd import lionmuon as lm

from parity import check_lion, check_muon

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    return t.detach().cpu().double().numpy()


def _state(shapes, seed):
    rng = np.random.default_rng(seed)
    W0 = [(rng.standard_normal(s) * 0.02).astype(np.float32) for s in shapes]
    M0 = [(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in shapes]
    G = [(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in shapes]
    return W0, M0, G


def _both(shapes, lion_only, seed, t, P, precision):
    """One step through lionmuon_step_ex and through lionmuon_step_noalloc on
    fresh copies of the same state; returns the inputs and both results."""
    W0, M0, G = _state(shapes, seed)
    cfg = lm.config(ns_precision=precision, lr_muon=0.02, lr_lion=1e-3)
    outs = []
    for noalloc in (False, True):
        W, M, Gd = [dev(x) for x in W0], [dev(x) for x in M0], [dev(x) for x in G]
        print(f"{'noalloc' if noalloc else 'step_ex'}: {len(shapes)} tensors t={t} P={P} "
              f"{precision}", flush=True)
        if noalloc:
            lm.lionmuon_step_noalloc(W, Gd, M, t, P, 0.9, 0.99, 0.1, cfg, lion_only=lion_only)
        else:
            lm.lionmuon_step_ex(W, Gd, M, t, P, 0.9, 0.99, 0.1, cfg, lion_only=lion_only)
        torch.cuda.synchronize()
        outs.append(([host(w) for w in W], [host(m) for m in M]))
    return W0, M0, G, outs


def _check(shapes, lion_only, seed, t, P, precision):
    W0, M0, G, outs = _both(shapes, lion_only, seed, t, P, precision)
    (wa, ma), (wb, mb) = outs
    for i in range(len(shapes)):
        assert np.array_equal(wa[i], wb[i]) and np.array_equal(ma[i], mb[i]), i
        muon = t % P == 0 if P else False
        if muon and min(shapes[i]) > 1 and not lion_only[i]:
            check_muon(W0[i], G[i], M0[i], wb[i], mb[i], 0.9, 0.99, 0.02, 0.1, precision)
        else:
            check_lion(W0[i], G[i], M0[i], wb[i], mb[i], 0.9, 0.99, 1e-3, 0.1)


def test_noalloc_matches_step_ex_on_consecutive_calls():
    big = [(768, 2304), (2304, 768), (1, 768), (300, 520)]
    small = [(256, 640), (1, 100)]
    # Muon step on the larger list, then on a smaller one (new tables), then a
    # Lion step and a Muon step on the larger list again (new addresses)
    _check(big, [False, False, False, False], 81, 0, 2, "bf16")
    _check(small, [False, False], 82, 0, 2, "bf16")
    _check(big, [False, False, False, True], 83, 1, 2, "bf16")
    _check(small, [False, False], 84, 3, 3, "fp32")


def test_noalloc_matches_step_ex_on_random_lists():
    """Twelve seeded random lists in a row (3-8 tensors of random shape and
    orientation, some 1-D or Lion-only; both precisions; Muon and Lion
    steps): every call rewrites the scratch's tables, and each result is
    bitwise that of lionmuon_step_ex and checked against the oracle."""
    rng = np.random.default_rng(86)
    done = 0
    for k in range(12):
        shapes, lion_only = [], []
        for _ in range(int(rng.integers(3, 9))):
            if rng.random() < 0.2:
                shapes.append((1, int(rng.integers(1, 3000))))
            else:
                s = int(rng.integers(2, 700))
                l = int(rng.integers(s, 1800))
                shapes.append((s, l) if rng.random() < 0.5 else (l, s))
            lion_only.append(bool(rng.random() < 0.15))
        precision = "fp32" if k % 4 == 3 else "bf16"
        t, P = (0, 2) if k % 3 else (1, 2)
        cfg = lm.config(ns_precision=precision)
        need = lm.lionmuon_workspace_bytes([(*sh, lo) for sh, lo in zip(shapes, lion_only)], cfg)
        if need > lm.NOALLOC_SCRATCH_BYTES - (4 << 20):    # room for the tables
            continue
        _check(shapes, lion_only, [87, k], t, P, precision)
        done += 1
    assert done >= 10


def test_noalloc_rejects_a_list_beyond_its_scratch():
    """A Muon step whose workspace exceeds the scratch is refused before
    anything is enqueued; a Lion step on the same list (no workspace) runs."""
    shapes = [(4096, 8192)]
    need = lm.lionmuon_workspace_bytes([(*s, False) for s in shapes])
    assert need > lm.NOALLOC_SCRATCH_BYTES
    W0, M0, G = _state(shapes, 85)
    W, M, Gd = [dev(x) for x in W0], [dev(x) for x in M0], [dev(x) for x in G]
    cfg = lm.config(lr_muon=0.02, lr_lion=1e-3)
    with pytest.raises(lm.LionMuonError) as e:
        lm.lionmuon_step_noalloc(W, Gd, M, 0, 1, 0.9, 0.99, 0.1, cfg)
    assert e.value.status == lm.LM_ERR_UNSUPPORTED and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert np.array_equal(host(W[0]), W0[0]) and np.array_equal(host(M[0]), M0[0])
    lm.lionmuon_step_noalloc(W, Gd, M, 1, 2, 0.9, 0.99, 0.1, cfg)
    torch.cuda.synchronize()
    rows = slice(0, 256)
    check_lion(W0[0][rows], G[0][rows], M0[0][rows], host(W[0])[rows], host(M[0])[rows],
               0.9, 0.99, 1e-3, 0.1)
