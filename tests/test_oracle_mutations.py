"""The oracle's pins catch planted mistakes (CPU only).

Each case below plants one plausible mistake into a copy of the oracle's
source (a flipped sign, a dropped term, a transposed operand, an index off by
one, a wrong scale, swapped blend weights), loads the copy as a separate
module, and runs every pin of tests/test_oracle_pins.py against it with all
of its parametrisations.  The unmodified copy must pass every pin; each
mutated copy must fail at least one.  Nothing here touches the real oracle
module or the GPU library.
"""

import itertools
import os
import types

import pytest

import test_oracle_pins as pins

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                          "oracle", "fmm_ref.py")

# (name, exact text in the oracle, replacement)
MUTATIONS = [
    ("phi_2 without the sign flip",
     "return _elu(-np.asarray(x, dtype=np.float64)) + 1.0",
     "return _elu(np.asarray(x, dtype=np.float64)) + 1.0"),
    ("elu without the -1",
     "np.expm1(np.minimum(x, 0.0))",
     "np.exp(np.minimum(x, 0.0))"),
    ("dense near field scaled by 1/d",
     'np.einsum("bhic,bhjc->bhij", q, k) / math.sqrt(d)',
     'np.einsum("bhic,bhjc->bhij", q, k) / d'),
    ("streamed near field without the scale",
     "    scale = 1.0 / math.sqrt(d)\n    out = np.empty_like(v)",
     "    scale = 1.0\n    out = np.empty_like(v)"),
    ("band one narrower",
     "return np.abs(i - j) <= band_k",
     "return np.abs(i - j) < band_k"),
    ("causal band without the diagonal",
     "return (j <= i) & (j >= i - band_k)",
     "return (j < i) & (j >= i - band_k)"),
    ("streamed band missing its last offset",
     "offs = np.arange(-kk, 1 if causal else kk + 1)",
     "offs = np.arange(-kk, 1 if causal else kk)"),
    ("far state transposed",
     's = np.einsum("bhjc,bhje->bhce", pk, v)',
     's = np.einsum("bhjc,bhje->bhec", pk, v)'),
    ("non-causal far part not normalised",
     "    for num, den in terms:\n        out += num / den[..., None]",
     "    for num, den in terms:\n        out += num / den.mean()"),
    ("causal far sum exclusive of j = i",
     "s_cum = s_run[:, :, None] + np.cumsum(outer, axis=2)",
     "s_cum = s_run[:, :, None] + np.cumsum(outer, axis=2) - outer"),
    ("causal far carry from the block's first row",
     "            s_run = s_cum[:, :, -1]",
     "            s_run = s_cum[:, :, 0]"),
    ("dense causal far triangle without the diagonal",
     "lower = np.tril(np.ones((n, n), dtype=bool))",
     "lower = np.tril(np.ones((n, n), dtype=bool), -1)"),
    ("blend weights swapped",
     "return np.where(a > 0, a * near, 0.0) + np.where(b > 0, b * far, 0.0)",
     "return np.where(a > 0, a * far, 0.0) + np.where(b > 0, b * near, 0.0)"),
    ("dense far field with one normaliser for both maps",
     "        w = a / a.sum(axis=-1, keepdims=True)",
     "        w = a / (rank * a.sum(axis=-1, keepdims=True).mean())"),
    ("rows form: causal band stops one short",
     "hi = i if causal else min(n - 1, i + band_k)",
     "hi = i - 1 if causal and i > 0 else min(n - 1, i + band_k)"),
    ("rows form: non-causal far state transposed",
     "            s = pk.T @ vs",
     "            s = (pk.T @ vs).T"),
    ("phi_3 not tanh",
     "return np.tanh(np.asarray(x, dtype=np.float64))",
     "return np.sin(np.asarray(x, dtype=np.float64))"),
    ("streamed joint far field with the denominators averaged",
     "        return num / den[..., None]",
     "        return num / (den[..., None] / len(terms))"),
    ("dense joint far field not row-normalised",
     "total / total.sum(axis=-1, keepdims=True), v)",
     "total, v)"),
    ("rows form: joint far field summed per map",
     "        far = sum(nums) / sum(dens)[:, None]",
     "        far = sum(nm / dn[:, None] for nm, dn in zip(nums, dens))"),
    ("backward: softmax derivative without the row term",
     "ds = p * (dp - gn[..., None])",
     "ds = p * dp"),
    ("backward: quotient rule with the wrong sign",
     "dden = -np.einsum(\"bhic,bhic->bhi\", f, num) / den ** 2",
     "dden = np.einsum(\"bhic,bhic->bhi\", f, num) / den ** 2"),
    ("backward: joint denominator squared",
     "dden = -np.einsum(\"bhic,bhic->bhi\", f, far) / den_all",
     "dden = -np.einsum(\"bhic,bhic->bhi\", f, far) / den_all ** 2"),
    ("backward: causal key gradients carried from the wrong end",
     "                ds_run = ds_suf[:, :, 0]",
     "                ds_run = ds_suf[:, :, -1]"),
    ("backward: phi_2 derivative without its sign",
     "return -np.where(-x > 0.0, 1.0, np.exp(np.minimum(-x, 0.0)))",
     "return np.where(-x > 0.0, 1.0, np.exp(np.minimum(-x, 0.0)))"),
    ("backward: sigmoid derivative missing its (1 - sigma)",
     "dw_near = sa * (1.0 - sa) * np.einsum",
     "dw_near = sa * np.einsum"),
    ("layer: heads taken d-major",
     "qkv = (x @ w_qkv).reshape(b_, n, 3, heads, d)",
     "qkv = (x @ w_qkv).reshape(b_, n, 3, d, heads).transpose(0, 1, 2, 4, 3)"),
    ("layer: heads merged in the wrong order",
     "merged = o.transpose(0, 2, 1, 3).reshape(b_, n, e)",
     "merged = o.transpose(0, 2, 3, 1).reshape(b_, n, e)"),
    ("fast weight: write without the read-back term",
     "w = w + beta[bb, hh, i] * np.outer(v[bb, hh, i] - u, pk[bb, hh, i])",
     "w = w + beta[bb, hh, i] * np.outer(v[bb, hh, i], pk[bb, hh, i])"),
    ("fast weight: keys not sum-normalised",
     "    pk = pk / pk.sum(axis=-1, keepdims=True)\n",
     "\n"),
    ("fast weight: normaliser updated after the output",
     "                z = z + pk[bb, hh, i]\n                out[bb, hh, i] = (w @ pq[bb, hh, i]) / (z @ pq[bb, hh, i])",
     "                out[bb, hh, i] = (w @ pq[bb, hh, i]) / ((z + 1e-30) @ pq[bb, hh, i])\n                z = z + pk[bb, hh, i]"),
    ("backward: key-side near gradient unscaled",
     "dk[:, :, j] += tau * ds[:, :, ok, t, None] * q[:, :, rows[ok]]",
     "dk[:, :, j] += ds[:, :, ok, t, None] * q[:, :, rows[ok]]"),
    ("fast-weight backward: W gradient not carried through the next write",
     "g_w = g_w - beta[bb, hh, i + 1] * np.outer(g_w @ p1, p1)",
     "g_w = g_w + 0.0 * beta[bb, hh, i + 1]"),
    ("fast-weight backward: key gradient reads W_i instead of W_{i-1}",
     "dpk[bb, hh, i] = beta[bb, hh, i] * (g_w.T @ e - wprev.T @ gp) + z_s",
     "dpk[bb, hh, i] = beta[bb, hh, i] * (g_w.T @ e - wi.T @ gp) + z_s"),
    ("fast-weight backward: normalisation derivative without the projection",
     "dk = phi_grad(k, 1) * (dpk - (dpk * pk).sum(axis=-1, keepdims=True)) / sk",
     "dk = phi_grad(k, 1) * dpk / sk"),
    ("layer backward: W_out gradient transposed",
     "    dw_out = m.T @ dyf\n",
     "    dw_out = (m.T @ dyf).T\n"),
    ("layer backward: x gradient through W_qkv untransposed",
     "    dx = (dqkv @ w_qkv.T).reshape(b_, n, e)",
     "    dx = (dqkv[:, :e] @ w_qkv[:, :e]).reshape(b_, n, e)"),
    ("fast-weight operator backward: linear part's gradients dropped",
     "        dq, dk, dv = dq + dql, dk + dkl, dv + dvl",
     "        dq, dk, dv = dq, dk, dv"),
]


def load_oracle(src: str) -> types.ModuleType:
    mod = types.ModuleType("oracle_copy")
    exec(compile(src, ORACLE_SRC + " (copy)", "exec"), mod.__dict__)
    return mod


def pin_calls():
    """Every pin test with every parametrisation, as (name, fn, kwargs)."""
    out = []
    for name in sorted(dir(pins)):
        fn = getattr(pins, name)
        if not name.startswith("test_") or not callable(fn):
            continue
        grids = []
        for mark in getattr(fn, "pytestmark", []):
            if mark.name != "parametrize":
                continue
            argnames, values = mark.args[0], mark.args[1]
            names = [a.strip() for a in argnames.split(",")] if isinstance(argnames, str) \
                else list(argnames)
            rows = [v if len(names) > 1 else (v,) for v in values]
            grids.append([dict(zip(names, r)) for r in rows])
        for combo in itertools.product(*grids) if grids else [()]:
            kw = {}
            for part in combo:
                kw.update(part)
            out.append((name, fn, kw))
    return out


def failing_pins(mod):
    saved = pins.ref
    pins.ref = mod
    failed = []
    try:
        for name, fn, kw in pin_calls():
            try:
                fn(**kw)
            except Exception:  # noqa: BLE001 - any failure counts as caught
                failed.append(f"{name}{kw or ''}")
    finally:
        pins.ref = saved
    return failed


def test_unmodified_copy_passes_every_pin():
    src = open(ORACLE_SRC).read()
    assert failing_pins(load_oracle(src)) == []


@pytest.mark.filterwarnings("ignore::RuntimeWarning")  # the broken copies divide by zero
@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new):
    src = open(ORACLE_SRC).read()
    assert src.count(old) == 1, f"mutation site for '{name}' must occur exactly once"
    failed = failing_pins(load_oracle(src.replace(old, new)))
    assert failed, f"no pin caught: {name}"
