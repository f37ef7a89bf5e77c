"""GPU <-> oracle parity of the split epoch kernel (kernel 9, long segments cut into parts) through
the C ABI.

Tolerances, as for the other epoch kernels:
  * after every epoch: |w - A model|_inf / |w|_inf <= 1e-4 with A model fresh in fp64;
  * one workgroup taking the units in order (window 1): the same visiting order as the oracle, so P
    within 1e-4 relative of the oracle's after every epoch (fp32 partial sums over parts of at most
    4,096 products, then over at most 256 parts);
  * asynchronous epochs, every epoch: gap <= 2 * oracle gap + 1e-6 P(0) (the fp32 floor); converged
    primal objective within 1e-5 relative;
  * the SVM box constraint exactly.
"""
import dataclasses

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as orc  # noqa: E402
from paper_1702_07005_amd import scd, synth  # noqa: E402

DEV = "cuda"
_cache = {}


def f64(t):
    return t.detach().cpu().numpy().astype(np.float64)


def fresh(p, model):
    return orc.fresh_shared(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, model)


def rel_inf(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))


def gap_gate(G, Gr, P0, where):
    floor = 1e-6 * abs(P0)
    assert G <= 2.0 * Gr + floor, (where, G, Gr, floor)


def oracle_curve(p, seed, n_epochs):
    model = np.zeros(p.C)
    shared = np.zeros(p.L)
    out = []
    for e in range(n_epochs):
        orc.epochs(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, seed, e, 1, model, shared)
        out.append(orc.objectives(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, model, shared))
    return model, shared, out


def transposed(p, form):
    # The CSC arrays of A (N x M) are the CSR arrays of its transpose (M x N): skewed rows.
    rng = np.random.default_rng(7)
    n = p.n_cols
    if form == "svm_dual":
        y = np.where(rng.random(n) < 0.5, -1.0, 1.0).astype(np.float32)
    else:
        y = rng.standard_normal(n).astype(np.float32)
    return dataclasses.replace(p, form=form, layout="csr", n_rows=n, n_cols=p.n_rows, y=y, lam=1.0 / n)


def ragged(form="ridge_primal"):
    """Segments of chosen lengths around multiples of 64 (the smallest part): empty ones (also the
    last, whose segment starts at nnz), 1, 63, 64, 65, ..., and one of exactly 256 parts of 64."""
    rng = np.random.default_rng(11)
    lens = [0, 1, 63, 64, 65, 127, 128, 129, 200, 640, 641, 1000, 4095, 4096, 4097, 16384, 3, 0]
    L = 20_000
    ptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    idx = np.concatenate([np.sort(rng.choice(L, n, replace=False)) for n in lens]).astype(np.int32)
    val = rng.standard_normal(int(ptr[-1])).astype(np.float32)
    C = len(lens)
    if form == "ridge_primal":
        y = rng.standard_normal(L).astype(np.float32)
        return synth.Problem("ragged", form, "csc", L, C, ptr, idx, val, y, 1.0 / L, 0)
    y = np.where(rng.random(C) < 0.5, -1.0, 1.0).astype(np.float32) if form == "svm_dual" else \
        rng.standard_normal(C).astype(np.float32)
    return synth.Problem("ragged", form, "csr", C, L, ptr, idx, val, y, 1.0 / C, 0)


def problem(key):
    if key in _cache:
        return _cache[key]
    if key == "text_ridge_twin":
        p = synth.make("text_ridge_csc", n_rows=3_500, n_cols=166_000, row_nnz=370)
    elif key == "text_ridge_long":  # columns beyond 4,096 entries
        p = synth.make("text_ridge_csc", n_rows=6_000, n_cols=166_000, row_nnz=370)
    elif key == "text_svm_twin":
        p = synth.make("text_svm", n_rows=3_500, n_cols=166_000, row_nnz=370)
    elif key == "dense_ridge":
        p = synth.make("dense_ridge")
    elif key == "svm_rows":
        p = transposed(problem("text_ridge_twin"), "svm_dual")
    elif key == "ridge_dual_rows":
        p = transposed(problem("text_ridge_twin"), "ridge_dual")
    elif key.startswith("ragged_"):
        p = ragged(key[len("ragged_"):])
    else:
        raise KeyError(key)
    _cache[key] = p
    return p


def forced(p, part, window, **opts):
    s = scd.solver_for(p)
    s.set_option("team", 0)
    s.set_option("hot", 0)
    for k, v in opts.items():
        s.set_option(k, v)
    s.set_option("window", window)
    s.set_option("split_part", part)
    s.set_option("split", 2)
    return s


# ---------------------------------------------------------------------------------- in order

IN_ORDER = {
    # (problem, part length, epochs)
    "dense_part64": ("dense_ridge", 64, 6),          # every column of 2,000 entries: 32 parts
    "dense_part4096": ("dense_ridge", 4096, 4),      # every column one FULL unit
    "text_ridge_part64": ("text_ridge_twin", 64, 3),  # up to 55 parts, most columns FULL
    "ragged_ridge": ("ragged_ridge_primal", 64, 4),
    "ragged_svm": ("ragged_svm_dual", 64, 4),
    "ragged_ridge_dual": ("ragged_ridge_dual", 64, 4),
    "svm_twin_part128": ("text_svm_twin", 128, 3),
}


@pytest.mark.parametrize("case", sorted(IN_ORDER))
def test_split_in_order_tracks_oracle(case):
    # One workgroup takes the units in order: GATHER parts, then the SCATTER parts that sum them,
    # coordinate after coordinate in permutation order -- the oracle's sequence, up to fp32 rounding.
    key, part, E = IN_ORDER[case]
    p = problem(key)
    _, _, curve = oracle_curve(p, 0, E)
    s = forced(p, part, 1)
    info = s.info()
    print(f"split in order {case}: kernel {info['kernel']} part {info['long_len']} window {info['window']}", flush=True)
    assert info["kernel"] == "split" and info["window"] == 1 and info["long_len"] == part
    for e in range(E):
        s.epochs(0, 1)
        P, _ = s.objective()
        Pr = curve[e][0]
        assert abs(P - Pr) <= 1e-4 * abs(Pr), (e, P, Pr)
        gm, gs, ep = s.get_state()
        model = f64(gm)
        assert ep == e + 1
        assert rel_inf(f64(gs), fresh(p, model)) <= 1e-4, e
        if p.form == "svm_dual":
            assert model.min() >= 0.0 and model.max() <= 1.0
    s.close()


def test_split_limits():
    p = problem("ragged_ridge_primal")  # longest segment 16,384 entries
    s = scd.solver_for(p)
    assert s.get_option("split") == 1 and s.get_option("split_part") == 0
    for k, bad in (("split", -1), ("split", 3), ("split_part", 63), ("split_part", 65), ("split_part", 4160),
                   ("split_part", -64)):
        with pytest.raises(scd.ScdError) as ei:
            s.set_option(k, bad)
        assert ei.value.code == -1
    s.set_option("window", 1)
    s.set_option("split_part", 64)  # 16,384 = 256 parts of 64: the most a segment may have
    s.set_option("split", 2)
    assert s.info()["kernel"] == "split"
    s.set_option("split_part", 0)
    assert s.info()["long_len"] == 4096
    s.close()
    # one entry more: 257 parts of 64, so the forced kernel is not taken
    q = dataclasses.replace(p, ptr=p.ptr.copy(), idx=p.idx.copy())
    lens = np.diff(q.ptr)
    j = int(np.argmax(lens))
    rng = np.random.default_rng(3)
    seg = set(q.idx[q.ptr[j]:q.ptr[j + 1]].tolist())
    extra = next(i for i in rng.permutation(q.n_rows) if i not in seg)
    col = np.sort(np.append(q.idx[q.ptr[j]:q.ptr[j + 1]], extra)).astype(np.int32)
    idx = np.concatenate([q.idx[:q.ptr[j]], col, q.idx[q.ptr[j + 1]:]]).astype(np.int32)
    val = np.concatenate([q.val[:q.ptr[j]], np.ones(1, np.float32), q.val[q.ptr[j]:]]).astype(np.float32)
    ptr = q.ptr.copy()
    ptr[j + 1:] += 1
    q = dataclasses.replace(q, ptr=ptr, idx=idx, val=val)
    t = scd.solver_for(q)
    t.set_option("window", 1)
    t.set_option("split_part", 64)
    t.set_option("split", 2)
    assert t.info()["max_segment"] == 16385 and t.info()["kernel"] != "split"
    t.close()


# ---------------------------------------------------------------------------------- asynchronous

ASYNC = {
    # (problem, part, window: 0 = automatic, extra options)
    "text_ridge_part256": ("text_ridge_twin", 256, 0, {}),
    "text_ridge_part64": ("text_ridge_twin", 64, 0, {}),
    "text_ridge_part256_fp64": ("text_ridge_twin", 256, 0, {"shared_fp64": 1}),
    "text_ridge_part256_chunk3": ("text_ridge_twin", 256, 0, {"queue_chunk": 3}),
    "text_ridge_part128_fresh": ("text_ridge_twin", 128, 0, {"fresh_reads": 1}),
    "svm_rows_part256": ("svm_rows", 256, 64, {}),
    "ridge_dual_rows_part256": ("ridge_dual_rows", 256, 64, {}),
    "dense_part512": ("dense_ridge", 512, 0, {}),
    "ragged_ridge_w4": ("ragged_ridge_primal", 64, 4, {}),
    "ragged_svm_w4": ("ragged_svm_dual", 64, 4, {}),
}


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("case", sorted(ASYNC))
def test_split_kernel_parity(case, seed):
    key, part, window, opts = ASYNC[case]
    p = problem(key)
    # The ragged matrices have 18 coordinates, so 4 in flight is far beyond any window the coupling
    # rule allows and single epochs are not comparable: there the gate is convergence after 40 epochs.
    ragged_case = key.startswith("ragged_")
    E = 40 if ragged_case else 6
    _, _, curve = oracle_curve(p, seed, E)
    s = forced(p, part, window, **opts)
    info = s.info()
    print(f"split {case} seed {seed}: kernel {info['kernel']} window {info['window']} part {info['long_len']}",
          flush=True)
    assert info["kernel"] == "split" and info["window"] == (window or info["auto_window"])
    P0, _ = s.objective()
    nonempty = np.diff(p.ptr) > 0
    prev = np.zeros(p.C)
    for e in range(E):
        s.epochs(seed, 1)
        gm, gs, _ = s.get_state()
        model = f64(gm)
        assert rel_inf(f64(gs), fresh(p, model)) <= 1e-4, e
        if p.form == "svm_dual":
            assert model.min() >= 0.0 and model.max() <= 1.0
        if e == 0 and p.form != "svm_dual":  # every coordinate was visited
            assert np.mean(model[nonempty] != prev[nonempty]) > 0.99, e
        prev = model
        G = s.duality_gap()
        print(f"  epoch {e + 1}: gap {G:.3e} oracle {curve[e][2]:.3e}", flush=True)
        if not ragged_case:
            gap_gate(G, curve[e][2], P0, e)
    if ragged_case:
        P, _ = s.objective()
        Pr, _, Gr = curve[-1]
        assert Gr <= 1e-7 * abs(Pr)  # the oracle has converged
        assert abs(P - Pr) <= 1e-5 * abs(Pr), (P, Pr)
    s.close()


def test_split_default_on_long_columns():
    # Columns beyond 4,096 entries: the automatic plan takes the split kernel at the full automatic
    # window (the queued kernel halves it); with the option off the queued kernel runs as before.
    p = problem("text_ridge_long")
    E = 6
    _, _, curve = oracle_curve(p, 0, E)
    s = scd.solver_for(p)
    info = s.info()
    print(f"text ridge long: kernel {info['kernel']} window {info['window']} auto {info['auto_window']} "
          f"max segment {info['max_segment']}", flush=True)
    assert info["max_segment"] > 4096 and info["kernel"] == "split" and info["long_len"] == 4096
    assert info["window"] == info["auto_window"]
    P0, _ = s.objective()
    for e in range(E):
        s.epochs(0, 1)
        gm, gs, _ = s.get_state()
        assert rel_inf(f64(gs), fresh(p, f64(gm))) <= 1e-4, e
        G = s.duality_gap()
        print(f"  epoch {e + 1}: gap {G:.3e} oracle {curve[e][2]:.3e}", flush=True)
        gap_gate(G, curve[e][2], P0, e)
    s.set_option("split", 0)
    info = s.info()
    assert info["kernel"] == "queued" and info["window"] == max(1, info["auto_window"] // 2)
    s.close()


@pytest.mark.parametrize("key,part,E", [("text_ridge_twin", 256, 40), ("dense_ridge", 512, 50)])
def test_split_converged_objective(key, part, E):
    # Run to convergence at the automatic window: primal objective within 1e-5 of the oracle's after
    # the same epochs (E: where the oracle's gap is below 1e-7 P); the dense workload also reaches
    # the normal-equation solution (Sec. II-A).
    p = problem(key)
    model = np.zeros(p.C)
    shared = np.zeros(p.L)
    orc.epochs(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 0, 0, E, model, shared)
    Pr, _, Gr = orc.objectives(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, model)
    assert Gr <= 1e-7 * abs(Pr)
    s = forced(p, part, 0)
    info = s.info()
    assert info["kernel"] == "split" and info["window"] > 1
    s.epochs(0, E)
    gm, gs, _ = s.get_state()
    beta = f64(gm)
    assert rel_inf(f64(gs), fresh(p, beta)) <= 1e-4
    P, _ = s.objective()
    print(f"split converged {key}: window {info['window']} P {P:.9e} oracle {Pr:.9e}", flush=True)
    assert abs(P - Pr) <= 1e-5 * abs(Pr), (P, Pr)
    if key == "dense_ridge":
        A = np.zeros((p.n_rows, p.n_cols))
        for m in range(p.n_cols):
            A[p.idx[p.ptr[m]:p.ptr[m + 1]], m] = p.val[p.ptr[m]:p.ptr[m + 1]]
        star = np.linalg.solve(A.T @ A + p.n_rows * p.lam * np.eye(p.n_cols), A.T @ p.y.astype(np.float64))
        assert rel_inf(beta, star) <= 1e-4, rel_inf(beta, star)
    s.close()


def test_split_wait_limit():
    # SCATTER units' bounded waits with a limit of one sleep: either every part's partials were in
    # time (valid state) or the timeout is reported at the next synchronising call and a written
    # state replaces the invalid one.
    p = problem("text_ridge_twin")
    s = forced(p, 64, 300)  # many workgroups, many parts: waits are likely to meet unpublished partials
    assert s.info()["kernel"] == "split"
    s.set_option("hot_wait_limit", 1)
    s.epochs(0, 2)
    try:
        s.duality_gap()
        timed_out = False
    except scd.ScdError as e:
        assert "timed out" in str(e)
        timed_out = True
    print(f"split wait limit 1: timed out {timed_out}", flush=True)
    if not timed_out:
        gm, gs, _ = s.get_state()
        assert rel_inf(f64(gs), fresh(p, f64(gm))) <= 1e-4
    s.set_option("hot_wait_limit", 0)
    s.set_state(torch.zeros(p.C, device=DEV), torch.zeros(p.L, device=DEV), 0)
    s.epochs(0, 2)
    gm, gs, _ = s.get_state()
    assert rel_inf(f64(gs), fresh(p, f64(gm))) <= 1e-4
    assert s.duality_gap() > 0.0
    s.close()
