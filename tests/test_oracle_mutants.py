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
