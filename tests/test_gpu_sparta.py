"""GPU parity of the sparse-averaging steps (section 4.2, Eq. (sparta) and
Eq. (delta_rule)) against the float64 oracle, through the C ABI binding.

Snapshots are copies and must be bit-exact.  The average and the delta rule
are float32 arithmetic: the bar is the fp32 parity bar (relative Frobenius
error <= 1e-5) plus a tighter bound from the arithmetic itself, and every
coordinate outside the round's positions must stay bit-identical.
"""
import numpy as np
import pytest
import torch

from helpers import TOL, rel
from oracle import ssn_oracle as O
from paper_2607_13332_amd import inputs as I
from paper_2607_13332_amd import ssn

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
# float32 sum of at most 64 weighted terms, one scaling, one subtraction:
# a few ulp per element, far below the parity bar.
AVG_BOUND = 2e-6
APPLY_BOUND = 2e-7


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    return t.detach().cpu().numpy()


def positions(n, m, form, seed):
    if form == "segment":
        first = (n - m) // 3
        return None, first, np.arange(first, first + m, dtype=np.int64)
    order = "sorted" if form == "sorted" else "random"
    p = I.sparta_positions_host(n, m, seed, order=order)
    return dev(p), 0, p


ROUND_CASES = [  # (n, m, R, form)
    (100_003, 5_000, 3, "segment"),
    (100_003, 4_999, 4, "segment"),    # ragged: scalar path
    (100_003, 5_000, 3, "sorted"),
    (100_003, 5_000, 5, "random"),
    (100_003, 4_998, 6, "sorted"),     # five to eight senders, scalar path
    (4_096, 1, 1, "segment"),
    (4_096, 4, 9, "random"),           # more senders than the register-held forms
    (257, 257, 64, "segment"),         # the whole vector, maximum sender count
]


@pytest.mark.parametrize("n,m,R,form", ROUND_CASES)
def test_round_against_oracle(n, m, R, form):
    """One round for every replica: snapshot, the reducer's weighted average
    with per-sender deltas, the receive step, then the delta rule applied to
    weights that moved on during the round."""
    seed = 1041 + n + m + R
    thetas = I.sparta_replicas_host(n, R, seed)
    Idev, first, P = positions(n, m, form, seed)
    print(f"[sparta] n={n} m={m} R={R} form={form}", flush=True)
    snaps = []
    for j in range(R):
        s = ssn.sparta_snapshot(dev(thetas[j]), I=Idev, first=first, m=m)
        assert np.array_equal(host(s), O.sparta_snapshot(thetas[j], P).astype(np.float32))
        snaps.append(s)
    w = [float(1 + (j % 3)) for j in range(R)]
    if R > 2:
        w[1] = 0.0                                  # a sender that absorbs the average
    acc, deltas = ssn.sparta_average(snaps, w)
    ref_acc, ref_deltas = O.sparta_average([host(s) for s in snaps], w)
    e = rel(host(acc), ref_acc)
    assert e <= min(TOL["f32"], AVG_BOUND), f"average rel {e:.3e}"
    for j in range(R):
        dl = host(deltas[j])
        # a delta can be exactly zero (one sender); compare against the
        # average's scale rather than the delta's own
        err = np.linalg.norm(dl - ref_deltas[j]) / max(np.linalg.norm(ref_acc), 1e-30)
        assert err <= AVG_BOUND, f"delta {j} error {err:.3e}"
    # receive: the buffer (holding the snapshot) plus the returned delta is
    # the average
    j = R - 1
    buf = dev(thetas[j])
    ssn.delta_rule(buf, deltas[j], None, I=Idev, first=first)
    got = host(buf)
    assert rel(got[P], ref_acc) <= AVG_BOUND
    mask = np.ones(n, bool)
    mask[P] = False
    assert np.array_equal(got[mask], thetas[j][mask])
    # apply: weights that advanced by `progress` during the round
    moved = (thetas[j] + I.sparta_progress_host(n, seed)).astype(np.float32)
    theta = dev(moved)
    ssn.delta_rule(theta, acc, snaps[j], I=Idev, first=first, lam=1.0)
    ref = O.delta_rule(moved, P, host(acc), host(snaps[j]), 1.0)
    got = host(theta)
    e = rel(got[P], ref[P])
    assert e <= APPLY_BOUND, f"delta rule rel {e:.3e}"
    assert np.array_equal(got[mask], moved[mask])


@pytest.mark.parametrize("lam", [0.0, 0.5, 1.0, 2.0])
def test_delta_rule_lambda(lam):
    """The AsyncMesh form: lam scales the correction; lam = 0 is a no-op."""
    n, m = 10_000, 2_048
    thetas = I.sparta_replicas_host(n, 2, 7)
    P = np.arange(100, 100 + m, dtype=np.int64)
    avg = thetas[1][P]
    snap = thetas[0][P] - 1e-3
    theta = dev(thetas[0])
    ssn.delta_rule(theta, dev(avg), dev(snap), first=100, lam=lam)
    ref = O.delta_rule(thetas[0], P, avg, snap, lam)
    got = host(theta)
    if lam == 0.0:
        assert np.array_equal(got, thetas[0])
    assert rel(got, ref) <= APPLY_BOUND


def test_vector_and_scalar_forms_agree_bitwise():
    """The 16-byte segment kernels and the per-element kernels do the same
    float32 operations in the same order."""
    n, m, R = 50_000, 4_096, 4
    thetas = I.sparta_replicas_host(n, R, 11)
    P = np.arange(1_000, 1_000 + m, dtype=np.int64)
    Pdev = dev(P)
    seg = [ssn.sparta_snapshot(dev(t), first=1_000, m=m) for t in thetas]
    lst = [ssn.sparta_snapshot(dev(t), I=Pdev) for t in thetas]
    for a, b in zip(seg, lst):
        assert torch.equal(a, b)
    acc_v, d_v = ssn.sparta_average(seg, [1.0, 2.0, 3.0, 0.5])
    # views offset by one element are 4-byte but not 16-byte aligned
    pad = [torch.cat([torch.zeros(1, device=DEV), s])[1:] for s in seg]
    acc_s = torch.empty(m + 1, device=DEV)[1:]
    acc_s, d_s = ssn.sparta_average(pad, [1.0, 2.0, 3.0, 0.5], acc=acc_s)
    assert torch.equal(acc_v, acc_s)
    for a, b in zip(d_v, d_s):
        assert torch.equal(a, b)
    t_v, t_s = dev(thetas[0]), dev(thetas[0])
    ssn.delta_rule(t_v, acc_v, seg[0], first=1_000)
    ssn.delta_rule(t_s, acc_v, seg[0], I=Pdev)
    assert torch.equal(t_v, t_s)


def test_twenty_rounds_reach_consensus():
    """Rounds rotate through 20 segments that tile the vector; replicas that
    do not move between rounds all hold the group average after a full pass
    (each round snapshot, average, apply on every replica)."""
    n, R = 40_001, 3
    thetas = I.sparta_replicas_host(n, R, 21)
    reps = [dev(t) for t in thetas]
    for r in range(I.SPARTA_TINY.segments):
        first, m = ssn.sparta_segment(n, r)
        snaps = [ssn.sparta_snapshot(t, first=first, m=m) for t in reps]
        acc, _ = ssn.sparta_average(snaps, deltas=False)
        for t, s in zip(reps, snaps):
            ssn.delta_rule(t, acc, s, first=first)
    ref = thetas.astype(np.float64).mean(axis=0)
    for t in reps:
        assert rel(host(t), ref) <= AVG_BOUND
    # snap + (avg - snap) is avg up to the rounding of the two float32 steps
    for t in reps[1:]:
        assert rel(host(t), host(reps[0])) <= APPLY_BOUND


def test_partial_delta_outputs_and_stream():
    """deltas=False and None entries skip those writes; a non-default stream
    gives the same result."""
    m = 1_000
    c = [dev(I.sparta_replicas_host(m, 1, 30 + r)[0]) for r in range(3)]
    d1 = torch.empty(m, device=DEV)
    acc, out = ssn.sparta_average(c, deltas=[None, d1, None])
    assert out[0] is None and out[2] is None
    ref_acc, ref_d = O.sparta_average([host(x) for x in c], [1.0, 1.0, 1.0])
    assert rel(host(d1), ref_d[1]) <= 1e-5
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        acc2, _ = ssn.sparta_average(c, deltas=False, stream=s)
    s.synchronize()
    assert torch.equal(acc, acc2)
    assert rel(host(acc), ref_acc) <= AVG_BOUND


def test_empty_round_is_a_no_op():
    theta = torch.ones(16, device=DEV)
    e = torch.empty(0, device=DEV)
    assert ssn.sparta_snapshot(theta, first=3, m=0).numel() == 0
    ssn.delta_rule(theta, e, e, first=16)
    assert torch.equal(theta, torch.ones(16, device=DEV))


def test_block8b_full_size_sampled():
    """The paper's per-block workload: 320M parameters, a 16M segment (round
    7 of the rotation) and a 16M random index set, four senders; checked on a
    seeded sample of positions that the oracle computes one by one, plus the
    untouched complement compared on the device."""
    cfg = I.SPARTA_BLOCK8B
    print(f"[sparta] {cfg.name} n={cfg.n} m={cfg.m} R={cfg.R}", flush=True)
    theta0 = I.sparta_replica_device(cfg.n, cfg.seed, DEV)
    sample = np.unique(np.concatenate([
        np.random.default_rng(5).choice(cfg.m, 4096, replace=False), [0, cfg.m - 1]]))
    sidx = torch.from_numpy(sample).to(DEV)
    for form in ("segment", "sorted"):
        if form == "segment":
            first, m = ssn.sparta_segment(cfg.n, 7)
            Idev = None
            pos = first + torch.arange(m, device=DEV, dtype=torch.int64)
        else:
            m = cfg.m
            first, Idev = 0, I.sparta_positions_device(cfg.n, m, cfg.seed, DEV)
            pos = Idev
        snap = ssn.sparta_snapshot(theta0, I=Idev, first=first, m=m)
        assert torch.equal(snap, theta0[pos])
        chunks = I.sparta_chunks_device(snap, cfg.R, cfg.seed)
        w = [1.0, 2.0, 0.0, 1.5]
        acc, deltas = ssn.sparta_average(chunks, w)
        cs = [host(c[sidx]) for c in chunks]
        ref_acc, ref_d = O.sparta_average(cs, w)
        assert rel(host(acc[sidx]), ref_acc) <= AVG_BOUND
        for j in range(cfg.R):
            err = np.linalg.norm(host(deltas[j][sidx]) - ref_d[j]) / np.linalg.norm(ref_acc)
            assert err <= AVG_BOUND
        theta = theta0 + 1e-3          # progress made while the round was in flight
        before = theta.clone()
        ssn.delta_rule(theta, acc, snap, I=Idev, first=first)
        ref = O.delta_rule(host(before[pos[sidx]]), np.arange(len(sample)),
                           host(acc[sidx]), host(snap[sidx]), 1.0)
        assert rel(host(theta[pos[sidx]]), ref) <= APPLY_BOUND
        keep = torch.ones(cfg.n, dtype=torch.bool, device=DEV)
        keep[pos] = False
        assert torch.equal(theta[keep], before[keep])
        del theta, before, keep, chunks, deltas, acc, snap, pos
        torch.cuda.empty_cache()
