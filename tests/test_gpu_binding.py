"""GPU tests of per-call tensor addresses, AdamW step counting and +-Inf
gradients, through the C ABI, against the fp64 oracle.

The library keeps one device plan per list signature (shapes, flags,
alignment) and uploads the call's tensor addresses separately, so buffers
that move between steps (fresh gradient tensors every step, weights copied
elsewhere) must give exactly the results of fixed buffers.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2605_19811_amd import lionmuon as lm

from parity import check_adamw, check_lion, check_muon

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

SHAPES = [(192, 320), (320, 192), (1, 700), (96, 130), (64, 64)]
LION_ONLY = [False, False, False, False, True]


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    return t.detach().cpu().double().numpy()


def _grad(seed, t, i, shape):
    return workloads.random_matrix([seed, t, i], *shape, std=1e-2)


def _initial(seed):
    W0 = [workloads.random_matrix([seed, 0, i], *s, std=0.02) for i, s in enumerate(SHAPES)]
    M0 = [workloads.random_matrix([seed, 1, i], *s, std=1e-2) for i, s in enumerate(SHAPES)]
    return W0, M0


def test_fresh_addresses_every_step_match_fixed_buffers():
    """Six steps (P = 2: Muon, Lion, ...): run A keeps one set of buffers
    and copies each gradient into it; run B hands the library freshly
    allocated gradient tensors every step (earlier ones kept alive, so every
    address is new) and moves W and M to new buffers before step 4. Each of
    B's steps is checked against the oracle from its pre-step state, and the
    two runs must agree bitwise."""
    seed = 71
    W0, M0 = _initial(seed)
    cfg = lm.config(ns_precision="bf16", lr_muon=0.02, lr_lion=1e-3)
    # run A: fixed addresses
    Wa, Ma = [dev(x) for x in W0], [dev(x) for x in M0]
    Ga = [torch.empty_like(w) for w in Wa]
    tl = lm.TensorList(Wa, Ga, Ma, LION_ONLY)
    for t in range(6):
        for i, s in enumerate(SHAPES):
            Ga[i].copy_(dev(_grad(seed, t, i, s)))
        lm.lionmuon_step_ex(None, None, None, t, 2, 0.9, 0.99, 0.1, cfg, tensors=tl)
    torch.cuda.synchronize()
    # run B: new gradient tensors every step, W and M moved once
    Wb, Mb = [dev(x) for x in W0], [dev(x) for x in M0]
    keep, seen = [], set()
    for t in range(6):
        if t == 4:
            keep.append((Wb, Mb))
            Wb, Mb = [w.clone() for w in Wb], [m.clone() for m in Mb]
        G = [_grad(seed, t, i, s) for i, s in enumerate(SHAPES)]
        Gb = [dev(g) for g in G]
        keep.append(Gb)
        addrs = {g.data_ptr() for g in Gb}
        assert not addrs & seen, "gradient addresses must be new"
        seen |= addrs
        before = [(host(w), host(m)) for w, m in zip(Wb, Mb)]
        print(f"fresh addresses: step {t}", flush=True)
        lm.lionmuon_step_ex(Wb, Gb, Mb, t, 2, 0.9, 0.99, 0.1, cfg, lion_only=LION_ONLY)
        torch.cuda.synchronize()
        for i in range(len(SHAPES)):
            w_prev, m_prev = before[i]
            if t % 2 == 0 and min(SHAPES[i]) > 1 and not LION_ONLY[i]:
                check_muon(w_prev, G[i], m_prev, host(Wb[i]), host(Mb[i]), 0.9, 0.99, 0.02, 0.1,
                           "bf16")
            else:
                check_lion(w_prev, G[i], m_prev, host(Wb[i]), host(Mb[i]), 0.9, 0.99, 1e-3, 0.1)
    for x, y in zip(Wa + Ma, Wb + Mb):
        assert torch.equal(x, y)


def test_alignment_class_change_between_calls():
    """The same shapes with 16-byte aligned buffers, then with buffers 4 bytes
    off (another plan: the per-element paths), then aligned again: every step
    matches the oracle."""
    seed = 72
    W0, M0 = _initial(seed)
    cfg = lm.config(ns_precision="fp32", lr_muon=0.02, lr_lion=1e-3)
    for t, off in enumerate([0, 1, 0, 1]):
        bufs = [[torch.zeros(int(np.prod(s)) + 8, device=DEV) for s in SHAPES] for _ in range(3)]
        W, M, Gd = ([b[off:off + int(np.prod(s))].view(s) for b, s in zip(bl, SHAPES)]
                    for bl in bufs)
        G = [_grad(seed, t, i, s) for i, s in enumerate(SHAPES)]
        for i in range(len(SHAPES)):
            W[i].copy_(dev(W0[i])); M[i].copy_(dev(M0[i])); Gd[i].copy_(dev(G[i]))
        P = 1 if t < 2 else 0                     # Muon steps, then Lion steps
        lm.lionmuon_step_ex(W, Gd, M, t, P, 0.9, 0.99, 0.1, cfg, lion_only=LION_ONLY)
        torch.cuda.synchronize()
        for i in range(len(SHAPES)):
            if P == 1 and min(SHAPES[i]) > 1 and not LION_ONLY[i]:
                check_muon(W0[i], G[i], M0[i], host(W[i]), host(M[i]), 0.9, 0.99, 0.02, 0.1, "fp32")
            else:
                check_lion(W0[i], G[i], M0[i], host(W[i]), host(M[i]), 0.9, 0.99, 1e-3, 0.1)


def test_one_plan_two_streams_different_addresses():
    """Two lists of one signature (so one cached plan) on two streams,
    enqueued back to back with caller workspaces and no host synchronisation:
    the second call rewrites the plan's address table, so it must first wait
    (on the device) for the first call's kernels."""
    shapes = [(768, 2304)] * 4 + [(1, 768)] * 4
    rng = np.random.default_rng(73)
    sets = []
    for _ in range(2):
        W0 = [(rng.standard_normal(s) * 0.02).astype(np.float32) for s in shapes]
        M0 = [(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in shapes]
        G = [(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in shapes]
        sets.append((W0, M0, G, [dev(x) for x in W0], [dev(x) for x in M0], [dev(x) for x in G]))
    cfg = lm.config(ns_precision="bf16", lr_muon=0.02, lr_lion=1e-3)
    nbytes = lm.lionmuon_workspace_bytes([(*s, False) for s in shapes], cfg)
    ws = [torch.empty(nbytes, dtype=torch.uint8, device=DEV) for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    print("one plan, two streams", flush=True)
    for k in range(2):
        _, _, _, W, M, G = sets[k]
        lm.lionmuon_step_ex(W, G, M, 0, 1, 0.9, 0.99, 0.1, cfg, workspace=ws[k],
                            stream=streams[k])
    torch.cuda.synchronize()
    for W0, M0, G, W, M, _ in sets:
        for i, s in enumerate(shapes):
            if s[0] > 1:
                check_muon(W0[i], G[i], M0[i], host(W[i]), host(M[i]), 0.9, 0.99, 0.02, 0.1, "bf16")
            else:
                check_lion(W0[i], G[i], M0[i], host(W[i]), host(M[i]), 0.9, 0.99, 1e-3, 0.1)


def test_adamw_step_count_zero_and_one_based_callers():
    """Four AdamW steps from zero moments, once with t = 0..3 and the
    default step count (t + 1), once with t = 1..4 and adam_step = t: both
    are AdamW steps 1..4 of the oracle, with identical results."""
    n = 5000
    W0 = workloads.random_matrix(74, 1, n, std=0.02)[0]
    runs = []
    for base in (0, 1):
        W, M, V = dev(W0), torch.zeros(n, device=DEV), torch.zeros(n, device=DEV)
        for k in range(4):
            t = base + k
            G = workloads.random_matrix([75, k], 1, n, std=1e-3)[0]
            cfg = lm.config(adam_step=t if base == 1 else 0)
            w_prev, m_prev, v_prev = host(W), host(M), host(V)
            lm.lionmuon_step_ex([W], [dev(G)], [M], t, 2, 0.9, 0.99, 0.1, cfg,
                                lion_only=[lm.LM_TENSOR_ADAMW], second_moment=[V])
            torch.cuda.synchronize()
            check_adamw(w_prev, G, m_prev, v_prev, host(W), host(M), host(V), k + 1, cfg)
        runs.append((W.cpu(), M.cpu(), V.cpu()))
    for x, y in zip(*runs):
        assert torch.equal(x, y)


def test_inf_gradients_propagate_like_the_oracle():
    """+-Inf gradient entries on both branches, no crash. Lion branch: Ghat
    is +-Inf there, so the update takes sign +-1 and W stays finite while M
    becomes +-Inf; an Inf meeting an Inf of the other sign in M makes both
    NaN. Muon branch: ||Ghat||_F is Inf, the normalised matrix holds NaN
    (Inf / Inf) where Ghat was infinite and 0 elsewhere, and NaN reaches every
    entry of the direction, as in the oracle."""
    rng = np.random.default_rng(76)
    shape = (64, 128)
    W0 = (rng.standard_normal(shape) * 0.02).astype(np.float32)
    M0 = (rng.standard_normal(shape) * 1e-2).astype(np.float32)
    G = (rng.standard_normal(shape) * 1e-2).astype(np.float32)
    G[3, 5], G[10, 20] = np.inf, -np.inf
    M0[10, 20] = np.inf                   # +Inf momentum meets a -Inf gradient
    for t, P in ((1, 2), (0, 2)):         # Lion step, then Muon step
        W, M = dev(W0), dev(M0)
        cfg = lm.config(ns_precision="fp32", lr_muon=0.01, lr_lion=0.01)
        print(f"Inf gradients, {'Muon' if t % P == 0 else 'Lion'} step", flush=True)
        lm.lionmuon_step_ex([W], [dev(G)], [M], t, P, 0.9, 0.99, 0.1, cfg)
        torch.cuda.synchronize()
        w_ref, m_ref = oracle.lionmuon_update(W0, G, M0, t, P, 0.9, 0.99, 0.01, 0.01, 0.1)
        w, m = host(W), host(M)
        for got, ref in ((w, w_ref), (m, m_ref)):
            assert np.array_equal(np.isnan(got), np.isnan(ref))
            assert np.array_equal(np.isposinf(got), np.isposinf(ref))
            assert np.array_equal(np.isneginf(got), np.isneginf(ref))
        assert np.isposinf(m[3, 5]) and np.isnan(m[10, 20])
        fin = np.isfinite(m_ref)
        assert np.abs(m[fin] - m_ref[fin]).max() <= 1e-6 * np.abs(m_ref[fin]).max()
        if t % P == 0:
            assert np.isnan(w).all()
        else:
            assert np.isfinite(w[3, 5]) and np.isnan(w[10, 20])
            fin = np.isfinite(w_ref)
            assert np.abs(w[fin] - w_ref[fin]).max() <= 1e-6 * np.abs(w_ref[fin]).max()


def test_plan_eviction_and_return():
    """Twenty lists of different signatures (more than the 16 cached plans),
    a Lion step each, then the first signature again (its plan was evicted and
    is rebuilt): every step matches the oracle."""
    rng = np.random.default_rng(77)
    shapes = [[(64 + 8 * i, 96), (1, 300 + i)] for i in range(20)] + [[(64, 96), (1, 300)]]
    for k, shp in enumerate(shapes):
        W0 = [(rng.standard_normal(s) * 0.02).astype(np.float32) for s in shp]
        M0 = [(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in shp]
        G = [(rng.standard_normal(s) * 1e-2).astype(np.float32) for s in shp]
        W, M = [dev(x) for x in W0], [dev(x) for x in M0]
        lm.lionmuon_step([W[0], W[1].view(-1)], [dev(G[0]), dev(G[1]).view(-1)],
                         [M[0], M[1].view(-1)], t=1, P=2, beta1=0.9, beta2=0.99, lr=0.01, wd=0.1)
        torch.cuda.synchronize()
        for i in range(2):
            check_lion(W0[i], G[i], M0[i], host(W[i]), host(M[i]), 0.9, 0.99, 0.01, 0.1)


def test_staging_ring_wraps_and_single_address_changes():
    """A list of 600 small tensors (19 KB of addresses per call) stepped 70
    times with one gradient tensor replaced by a fresh one on every call, so
    the address table is rewritten each time and the 1 MB staging ring wraps
    around; every tensor is checked on the last calls."""
    n = 600
    rng = np.random.default_rng(78)
    sizes = [int(rng.integers(1, 300)) for _ in range(n)]
    W0 = [(rng.standard_normal(k) * 0.02).astype(np.float32) for k in sizes]
    M0 = [(rng.standard_normal(k) * 1e-2).astype(np.float32) for k in sizes]
    G = [(rng.standard_normal(k) * 1e-2).astype(np.float32) for k in sizes]
    Gd = [dev(g) for g in G]
    keep = []
    for call in range(70):
        W, M = [dev(x) for x in W0], [dev(x) for x in M0]
        j = call % n
        fresh = dev(G[j])                          # new address for tensor j only
        keep.append(fresh)
        grads = list(Gd)
        grads[j] = fresh
        lm.lionmuon_step(W, grads, M, t=1, P=2, beta1=0.9, beta2=0.99, lr=0.01, wd=0.1)
        if call >= 67:
            torch.cuda.synchronize()
            for i in range(n):
                check_lion(W0[i], G[i], M0[i], host(W[i]), host(M[i]), 0.9, 0.99, 0.01, 0.1)
