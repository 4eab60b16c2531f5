"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each case swaps one piece of the oracle for a plausible wrong variant and
checks that an independent pin (brute force, closed form, golden code
table) no longer agrees.
"""
import numpy as np
import pytest

from oracle import brute, formats, paged


def _case():
    rng = np.random.default_rng(21)
    ps, Hq, Hkv, D = 2, 4, 2, 8
    P, n = [9], [4]
    npg = -(-(P[0] + n[0]) // ps)
    bt = rng.permutation(npg + 1)[:npg].astype(np.int32)[None]
    pk = rng.standard_normal((npg + 1, Hkv, ps, D)).astype(np.float32)
    pv = rng.standard_normal((npg + 1, Hkv, ps, D)).astype(np.float32)
    q = rng.standard_normal((4, Hq, D)).astype(np.float32)
    return q, pk, pv, bt, P, n, ps


def _gap(window):
    q, pk, pv, bt, P, n, ps = _case()
    out = paged.prefix_prefill(q, pk, pv, bt, np.array(P), np.array(n), page_size=ps,
                               kv_dtype="f32", softmax_scale=0.3, window=window)
    ref = brute.prefill(q.astype(np.float64).tolist(), pk.astype(np.float64).tolist(),
                        pv.astype(np.float64).tolist(), bt.tolist(), P, n, ps, 0.3, window)
    return np.max(np.abs(out - np.array(ref)))


def test_unmutated_oracle_agrees():
    assert _gap(0) <= 1e-12 and _gap(3) <= 1e-12


@pytest.mark.parametrize("mutant", [
    lambda i, j, W: (j < i) | (j == i) & False,            # drops the diagonal key
    lambda i, j, W: (j <= i) & ((W <= 0) | (i - j <= W)),  # window one key too wide
    lambda i, j, W: (j <= i + 1) & ((W <= 0) | (i - j < W)),  # sees one future key
])
def test_visibility_mutants_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(paged, "visible", mutant)
    assert max(_gap(0), _gap(3)) > 1e-6


def test_head_mapping_mutant_is_caught(monkeypatch):
    real = paged.attend

    def modulo_heads(q, pos, k, v, scale, window=0, row_chunk=None):
        # query head h reading KV head h % H_kv instead of h // G
        Hkv = k.shape[1]
        G = q.shape[1] // Hkv
        order = np.array([(h % Hkv) * G + h // Hkv for h in range(q.shape[1])])
        inv = np.argsort(order)
        return real(q[:, inv], pos, k, v, scale, window, row_chunk)[:, order]

    monkeypatch.setattr(paged, "attend", modulo_heads)
    assert _gap(0) > 1e-6


def test_rounding_mutant_is_caught(monkeypatch):
    real = formats.e4m3_encode

    def ties_away(r):
        r = np.asarray(r, dtype=np.float64)
        bumped = r + np.sign(r) * np.spacing(np.abs(r))  # nudges ties upward
        return real(np.clip(bumped, -448, 448))

    monkeypatch.setattr(formats, "e4m3_encode", ties_away)
    assert formats.e4m3_encode(np.float64(1.0625)) != 0x38


def test_dropped_max_subtraction_overflows_where_oracle_does_not():
    # logits near 1000 overflow exp() without the maximum subtraction; the
    # oracle subtracts it and stays finite
    k = np.zeros((3, 1, 2))
    k[:, 0, 0] = [1000.0, 1001.0, 999.0]
    v = np.arange(6, dtype=np.float64).reshape(3, 1, 2)
    q = np.array([[[1.0, 0.0]]])
    out = paged.attend(q, np.array([2]), k, v, 1.0, 0)
    w = np.exp(np.array([1000.0, 1001.0, 999.0]) - 1001.0)
    assert np.allclose(out[0, 0], (w @ v[:, 0]) / w.sum(), atol=1e-14)


# ---------------------------------------------------------------- TTL oracle

def _ttl_pins_hold():
    """The TTL oracle's worked examples and closed forms (see test_ttl.py)."""
    import math

    from oracle import ttl

    grid = np.linspace(0.0, 12.0, 12001)
    ok = ttl.eq2_ttl([1.0, 2.0, 3.0, 10.0], 5.0) == 3.0
    ok &= ttl.eq2_ttl([1.0, 1.0, 1.0, 4.0], 2.0) == 1.0
    ok &= ttl.eq2_ttl([2.0, 4.0], 4.0) == 0.0
    for B in (0.5, 2.0, 10.0):
        best = grid[np.argmax((1.0 - np.exp(-grid)) * B - grid)]
        ok &= abs(ttl.cold_ttl(B) - best) < 2e-3
    ok &= abs(ttl.memoryfulness([5] * 10) - 1.0) < 1e-12
    ok &= abs(ttl.memoryfulness([1, 3]) - 5.0 / 11.0) < 1e-12
    return bool(ok) and math.isfinite(ttl.cold_ttl(2.0))


def test_unmutated_ttl_oracle_agrees():
    assert _ttl_pins_hold()


@pytest.mark.parametrize("name, mutant", [
    ("cdf", lambda S, tau: sum(1 for t in S if t < tau) / len(S)),          # strict: misses the step
    ("cold_ttl", lambda B: max(0.0, np.log(B) - 1.0) if B > 0 else 0.0),      # shifted optimum
    ("cold_ttl", lambda B: max(0.0, np.log(2.0 * B)) if B > 0 else 0.0),      # lost factor
])
def test_ttl_formula_mutants_are_caught(monkeypatch, name, mutant):
    from oracle import ttl

    monkeypatch.setattr(ttl, name, mutant)
    assert not _ttl_pins_hold()


def test_memoryfulness_sign_mutant_is_caught(monkeypatch):
    from oracle import ttl

    real = ttl.memoryfulness
    monkeypatch.setattr(ttl, "memoryfulness", lambda Ns: -real(Ns))   # Corr instead of -Corr
    assert not _ttl_pins_hold()


def test_eq2_candidate_mutant_is_caught(monkeypatch):
    from oracle import ttl

    def no_zero(S, B):  # forgets the tau = 0 candidate
        best_tau, best = None, None
        for tau in sorted(set(S)):
            val = ttl.cdf(S, tau) * B - tau
            if best is None or val > best:
                best_tau, best = tau, val
        return best_tau

    monkeypatch.setattr(ttl, "eq2_ttl", no_zero)
    assert not _ttl_pins_hold()
