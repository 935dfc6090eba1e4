"""Pins for the CPU float64 oracle (no GPU).

The paper prints no attention values, so the oracle is pinned to facts that do
not come from the oracle itself: central finite differences of the loss
l = <O, dO>, closed forms, exact invariants, a metamorphic shift, permutation
equivariance, and an independent derivation (PyTorch autograd through its own
softmax / scaled_dot_product_attention), which is how the paper's kernels were
verified (abstract; section sec:methodology, "Kernels benchmarked"). The last
test plants typical mistakes in the oracle and checks that a pin catches each.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import naive as orc




def _rand(rng, *shape, scale=1.0):
    return rng.standard_normal(shape) * scale


def _loss(q, k, v, do, s, causal):
    _, _, O, _ = orc.forward_head(q, k, v, s, causal)
    return float((O * do).sum())


def _fd_grads(q, k, v, do, s, causal, h=1e-6):
    """Central differences of l = <O, dO> with respect to Q, K and V."""
    grads = []
    for which in range(3):
        X = [q, k, v][which]
        G = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            args_p = [q.copy(), k.copy(), v.copy()]
            args_m = [q.copy(), k.copy(), v.copy()]
            args_p[which][idx] += h
            args_m[which][idx] -= h
            G[idx] = (_loss(*args_p, do, s, causal) - _loss(*args_m, do, s, causal)) / (2 * h)
        grads.append(G)
    return grads


FD_CASES = [(1, 3, False), (3, 2, False), (5, 3, True), (4, 2, True), (6, 4, False), (7, 3, True)]


@pytest.mark.parametrize("n,d,causal", FD_CASES)
def test_gradients_match_central_differences(n, d, causal):
    rng = np.random.default_rng(100 + 10 * n + d)
    q, k, v, do = (_rand(rng, n, d) for _ in range(4))
    s = 0.7
    r = orc.attention_head(q, k, v, do, s, causal)
    gq, gk, gv = _fd_grads(q, k, v, do, s, causal)
    for name, G, ref in (("dQ", r["dQ"], gq), ("dK", r["dK"], gk), ("dV", r["dV"], gv)):
        np.testing.assert_allclose(G, ref, rtol=1e-6, atol=1e-8, err_msg=name)


@pytest.mark.parametrize("causal", [False, True])
def test_softmax_and_score_gradient_rows(causal):
    rng = np.random.default_rng(7)
    n, d = 37, 8
    q, k, v, do = (_rand(rng, n, d) for _ in range(4))
    r = orc.attention_head(q, k, v, do, 1 / math.sqrt(d), causal, keep=True)
    p_err, ds_err = orc.row_invariants(r["P"], r["dS"])
    assert p_err <= 1e-12
    assert ds_err <= 1e-12
    if causal:
        # masked probabilities, hence masked score gradients, are exactly zero
        upper = np.triu(np.ones((n, n), dtype=bool), k=1)
        assert np.all(r["P"][upper] == 0.0)
        assert np.all(r["dS"][upper] == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_constant_values_closed_form(causal):
    """Every value row equal to v: O_i = v for all i, and dQ = dK = 0 because
    each row of dP is constant, so dP - D vanishes."""
    rng = np.random.default_rng(11)
    n, d = 19, 5
    q, k, do = (_rand(rng, n, d) for _ in range(3))
    vrow = _rand(rng, d)
    v = np.tile(vrow, (n, 1))
    r = orc.attention_head(q, k, v, do, 0.5, causal)
    np.testing.assert_allclose(r["O"], v, rtol=0, atol=1e-14)
    assert np.abs(r["dQ"]).max() <= 1e-13
    assert np.abs(r["dK"]).max() <= 1e-13


def test_single_key_closed_form():
    """n = 1: P = 1, O = v_0, L = s q.k, no gradient reaches Q or K, dV = dO."""
    rng = np.random.default_rng(12)
    d = 6
    q, k, v, do = (_rand(rng, 1, d) for _ in range(4))
    s = 0.3
    r = orc.attention_head(q, k, v, do, s, causal=False)
    np.testing.assert_allclose(r["O"], v, rtol=0, atol=1e-15)
    np.testing.assert_allclose(r["L"], [s * float(q[0] @ k[0])], rtol=1e-15)
    np.testing.assert_array_equal(r["dQ"], 0.0)
    np.testing.assert_array_equal(r["dK"], 0.0)
    np.testing.assert_allclose(r["dV"], do, rtol=0, atol=1e-15)


@pytest.mark.parametrize("causal", [False, True])
def test_zero_queries_closed_form(causal):
    """Q = 0: every unmasked score is 0, so P is uniform over the kept keys.
    O_i is the mean of v_j (the prefix mean j <= i with the causal mask) and
    L_i = ln n (ln(i + 1) with the causal mask)."""
    rng = np.random.default_rng(13)
    n, d = 23, 4
    k, v, do = (_rand(rng, n, d) for _ in range(3))
    q = np.zeros((n, d))
    r = orc.attention_head(q, k, v, do, 0.9, causal)
    if causal:
        counts = np.arange(1, n + 1)
        mean = np.cumsum(v, axis=0) / counts[:, None]
        np.testing.assert_allclose(r["L"], np.log(counts), rtol=1e-15, atol=1e-15)
    else:
        mean = np.tile(v.mean(axis=0), (n, 1))
        np.testing.assert_allclose(r["L"], np.full(n, math.log(n)), rtol=1e-15)
    np.testing.assert_allclose(r["O"], mean, rtol=1e-13, atol=1e-14)


def test_two_keys_logistic_closed_form():
    """d = 1, two keys: P_i0 = logistic(s q_i (k_0 - k_1)), so
    O_i = v_1 + logistic(.) (v_0 - v_1) and L_i = log(e^{s q_i k_0} + e^{s q_i k_1})."""
    q = np.array([[0.5], [-2.0], [1.25]])
    k = np.array([[1.5], [-0.75]])
    v = np.array([[3.0], [-1.0]])
    s = 0.8
    # three queries against two keys: pad to a square problem by repeating keys
    # is not needed -- the oracle's forward accepts n_q != n_k when non-causal
    _, P, O, L = orc.forward_head(q, k, v, s, causal=False)
    for i in range(3):
        z = s * q[i, 0] * (k[0, 0] - k[1, 0])
        p0 = 1.0 / (1.0 + math.exp(-z))
        assert abs(P[i, 0] - p0) <= 1e-15
        assert abs(O[i, 0] - (v[1, 0] + p0 * (v[0, 0] - v[1, 0]))) <= 1e-14
        ref_L = math.log(math.exp(s * q[i, 0] * k[0, 0]) + math.exp(s * q[i, 0] * k[1, 0]))
        assert abs(L[i] - ref_L) <= 1e-14


def test_causal_first_row_attends_only_to_itself():
    rng = np.random.default_rng(14)
    n, d = 9, 3
    q, k, v, do = (_rand(rng, n, d) for _ in range(4))
    s = 0.6
    r = orc.attention_head(q, k, v, do, s, causal=True, keep=True)
    assert r["P"][0, 0] == 1.0
    np.testing.assert_allclose(r["O"][0], v[0], rtol=0, atol=1e-15)
    assert abs(r["L"][0] - s * float(q[0] @ k[0])) <= 1e-14


@pytest.mark.parametrize("causal", [False, True])
def test_key_shift_metamorphic(causal):
    """K -> K + 1 c^T adds s q_i.c to row i of S: P, O, dV, dK are unchanged,
    L_i shifts by s q_i.c, and dQ is unchanged because rows of dS sum to 0."""
    rng = np.random.default_rng(15)
    n, d = 17, 6
    q, k, v, do = (_rand(rng, n, d) for _ in range(4))
    c = _rand(rng, d)
    s = 0.45
    a = orc.attention_head(q, k, v, do, s, causal)
    b = orc.attention_head(q, k + c[None, :], v, do, s, causal)
    for key in ("O", "dQ", "dK", "dV"):
        np.testing.assert_allclose(b[key], a[key], rtol=1e-10, atol=1e-12, err_msg=key)
    np.testing.assert_allclose(b["L"], a["L"] + s * (q @ c), rtol=1e-12, atol=1e-12)


def test_permutation_equivariance_non_causal():
    rng = np.random.default_rng(16)
    n, d = 15, 4
    q, k, v, do = (_rand(rng, n, d) for _ in range(4))
    s = 0.5
    a = orc.attention_head(q, k, v, do, s, False)
    pk = rng.permutation(n)
    b = orc.attention_head(q, k[pk], v[pk], do, s, False)
    for key in ("O", "L", "dQ"):
        np.testing.assert_allclose(b[key], a[key], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(b["dK"], a["dK"][pk], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(b["dV"], a["dV"][pk], rtol=1e-12, atol=1e-13)
    pq = rng.permutation(n)
    c = orc.attention_head(q[pq], k, v, do[pq], s, False)
    for key in ("O", "L", "dQ"):
        np.testing.assert_allclose(c[key], a[key][pq], rtol=1e-12, atol=1e-13)
    for key in ("dK", "dV"):
        np.testing.assert_allclose(c[key], a[key], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_whole_tensor_invariants(causal):
    """Identities that hold for every head at any size; the GPU tests apply
    them to full-size outputs: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i,
    <Q, dQ> = <K, dK>, <V, dV> = <O, dO>."""
    rng = np.random.default_rng(17)
    n, d = 41, 8
    q, k, v, do = (_rand(rng, n, d) for _ in range(4))
    r = orc.attention_head(q, k, v, do, 1 / math.sqrt(d), causal)
    assert np.abs(r["dK"].sum(axis=0)).max() <= 1e-12
    np.testing.assert_allclose(r["dV"].sum(axis=0), do.sum(axis=0), rtol=1e-12, atol=1e-12)
    assert abs(float((q * r["dQ"]).sum()) - float((k * r["dK"]).sum())) <= 1e-12
    assert abs(float((v * r["dV"]).sum()) - float((r["O"] * do).sum())) <= 1e-12


@pytest.mark.parametrize("causal", [False, True])
def test_matches_torch_autograd_float64(causal):
    """Independent derivation: PyTorch's own scaled_dot_product_attention
    (math path) and autograd, in float64 on the CPU."""
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F

    rng = np.random.default_rng(18)
    B, H, n, d = 2, 3, 33, 16
    q, k, v, do = (_rand(rng, B, H, n, d) for _ in range(4))
    s = 1 / math.sqrt(d)
    r = oracle.attention(q, k, v, do, s, causal)
    tq, tk, tv = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v))
    out = F.scaled_dot_product_attention(tq, tk, tv, is_causal=causal, scale=s)
    out.backward(torch.tensor(do, dtype=torch.float64))
    np.testing.assert_allclose(r["O"], out.detach().numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r["dQ"], tq.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(r["dK"], tk.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(r["dV"], tv.grad.numpy(), rtol=1e-10, atol=1e-12)
    logits = s * torch.tensor(q) @ torch.tensor(k).transpose(-1, -2)
    if causal:
        logits = logits.masked_fill(torch.ones(n, n, dtype=torch.bool).triu(1), float("-inf"))
    np.testing.assert_allclose(r["L"], torch.logsumexp(logits, dim=-1).numpy(), rtol=1e-13, atol=1e-13)


def test_forward_only_and_row_sampler_agree_with_full():
    rng = np.random.default_rng(19)
    B, H, n, d = 1, 2, 29, 8
    q, k, v, do = (_rand(rng, B, H, n, d) for _ in range(4))
    s = 0.35
    for causal in (False, True):
        full = oracle.attention(q, k, v, do, s, causal)
        fwd = oracle.attention_forward(q, k, v, s, causal)
        np.testing.assert_array_equal(fwd["O"], full["O"])
        np.testing.assert_array_equal(fwd["L"], full["L"])
        rows = np.array([0, 5, 28])
        sub = oracle.rows_forward_dq(q[0, 1], k[0, 1], v[0, 1], do[0, 1], rows, s, causal)
        for key in ("O", "L", "dQ"):
            np.testing.assert_allclose(sub[key], full[key][0, 1][rows], rtol=1e-13, atol=1e-14)
        heads = [(0, 1)]
        part = oracle.attention(q, k, v, do, s, causal, heads=heads)
        np.testing.assert_array_equal(part["dK"][0], full["dK"][0, 1])


def test_max_rel_err_definition():
    ref = np.array([1.0, -4.0, 2.0])
    x = np.array([1.1, -4.0, 1.8])
    assert orc.max_rel_err(x, ref) == pytest.approx(0.2 / 4.0)
    assert orc.max_rel_err(np.zeros(2), np.zeros(2)) == 0.0


# --- planted mistakes: each must be caught by at least one pin -------------

def _pins_pass(mod):
    """Run a compact subset of the pins against ``mod`` (the oracle module,
    possibly with a planted mistake); return True when all of them pass."""
    try:
        rng = np.random.default_rng(5)
        for (n, d, causal) in [(4, 3, True), (3, 2, False)]:
            q, k, v, do = (_rand(rng, n, d) for _ in range(4))
            s = 0.7
            r = mod.attention_head(q, k, v, do, s, causal)
            gq, gk, gv = _fd_grads(q, k, v, do, s, causal)
            for G, ref in ((r["dQ"], gq), (r["dK"], gk), (r["dV"], gv)):
                if not np.allclose(G, ref, rtol=1e-6, atol=1e-8):
                    return False
        n, d = 11, 3
        k, v, do = (_rand(rng, n, d) for _ in range(3))
        for causal in (False, True):
            r = mod.attention_head(np.zeros((n, d)), k, v, do, 0.9, causal)
            cnt = np.arange(1, n + 1) if causal else np.full(n, n)
            mean = np.cumsum(v, axis=0) / cnt[:, None] if causal else np.tile(v.mean(0), (n, 1))
            if not (np.allclose(r["L"], np.log(cnt)) and np.allclose(r["O"], mean)):
                return False
        return True
    except (FloatingPointError, ValueError):
        return False


def test_unmodified_oracle_passes_pin_subset():
    assert _pins_pass(orc)


MUTANTS = {
    # dQ without the score scale
    "dq_scale": lambda q, k, v, do, P, s: (lambda r: (r[0] / s,) + r[1:])(_REAL_BWD(q, k, v, do, P, s)),
    # dK from dS instead of dS^T (a transposed operand)
    "dk_transpose": lambda q, k, v, do, P, s: (lambda r: (r[0], s * (r[3] @ np.asarray(q, float)),) + r[2:])(_REAL_BWD(q, k, v, do, P, s)),
    # sign of the score gradient flipped
    "ds_sign": lambda q, k, v, do, P, s: (lambda r: (-r[0], -r[1]) + r[2:])(_REAL_BWD(q, k, v, do, P, s)),
    # dV from P instead of P^T
    "dv_transpose": lambda q, k, v, do, P, s: (lambda r: (r[0], r[1], P @ np.asarray(do, float)) + r[3:])(_REAL_BWD(q, k, v, do, P, s)),
}
_REAL_BWD = orc.backward_head


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_backward_mistakes_are_caught(monkeypatch, name):
    monkeypatch.setattr(orc, "backward_head", MUTANTS[name])
    assert not _pins_pass(orc)


def test_planted_mask_off_by_one_is_caught(monkeypatch):
    real_scores = orc.scores

    def shifted(q, k, scale, causal):
        S = real_scores(q, k, scale, False)
        if causal:
            n_q, n_k = S.shape
            S[np.triu(np.ones((n_q, n_k), dtype=bool), k=2)] = -np.inf  # keeps key i+1
        return S

    monkeypatch.setattr(orc, "scores", shifted)
    assert not _pins_pass(orc)


def test_planted_log_base_mistake_is_caught(monkeypatch):
    real_fwd = orc.forward_head

    def log2_lse(q, k, v, scale, causal):
        S, P, O, L = real_fwd(q, k, v, scale, causal)
        return S, P, O, L / math.log(2.0)

    monkeypatch.setattr(orc, "forward_head", log2_lse)
    assert not _pins_pass(orc)
