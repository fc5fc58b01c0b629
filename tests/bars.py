"""Parity bars for gradients that are sums over many terms (MLP weights, gate logits).

Such a gradient is compared as a whole tensor: max |gpu - oracle| / max |oracle| must stay
under the storage type's bar (2e-2 bf16, 1e-4 f32), the output bar relative to the
gradient's own scale. A zeroed, sign-flipped or badly scaled gradient therefore fails
(its error is the gradient's own maximum, or twice it), as does a few-percent error on
its largest entries.

Two kinds of gradient have no scale of their own and are bounded differently:
  * identically zero by the method's algebra: the key MLP's output bias b2. A common
    shift of every compressed key adds the same amount to every score of a query
    (Eq. 5 attention), which the softmax ignores, so the bias's summed terms cancel
    exactly. Its value on either side is rounding of that cancellation; it is bounded
    per entry by the bar times the magnitude of its summed terms (sum of |term|, the
    error bound of a sum), and the oracle's own value must vanish to float64 rounding;
  * every term zero (no compressed key with a gradient, e.g. a single real point whose
    softmax over one eligible compressed key is constant): bounded absolutely at 1e-6.
"""
from __future__ import annotations

import numpy as np

ABS_ZERO = 1e-6      # absolute bound where every term of the oracle's sum vanishes

# gradients that vanish identically by the softmax's shift invariance
IDENTICALLY_ZERO = {"dphi_k.b2"}


def summed_error(name: str, gpu, ref, terms) -> tuple[str, float]:
    """(kind, error) of one summed gradient against the oracle; see the module text.

    kind is "rel" (max-abs over max |oracle|), "cancel" (per entry over sum |term|) or
    "abs" (absolute, every term zero)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    terms = np.asarray(terms, np.float64)
    assert gpu.shape == ref.shape == terms.shape, (name, gpu.shape, ref.shape, terms.shape)
    tmax = float(terms.max()) if terms.size else 0.0
    if tmax < 1e-12:
        return "abs", float(np.abs(gpu).max()) if gpu.size else 0.0
    if name in IDENTICALLY_ZERO:
        # the oracle's value is float64 rounding of an exact cancellation
        assert float(np.abs(ref).max()) <= 1e-9 * tmax, (name, float(np.abs(ref).max()), tmax)
        return "cancel", float(np.max(np.abs(gpu - ref) / np.maximum(terms, 1e-30)))
    rmax = float(np.abs(ref).max())
    assert rmax > 1e-9 * tmax, f"{name}: oracle gradient vanishes against its terms; not a known zero"
    return "rel", float(np.abs(gpu - ref).max() / rmax)


def summed_ok(kind: str, err: float, tol: float) -> bool:
    return err < (ABS_ZERO if kind == "abs" else tol)


def check_summed(grads: dict, ref: dict, tol: float) -> dict:
    """Compare every summed gradient; grads/ref map names ("dgate", "dphi_k.w1", ...) to
    arrays, ref["abs"] to their term magnitudes. Returns {name: (kind, err)} and asserts
    each bar."""
    out = {}
    for name, g in grads.items():
        kind, err = summed_error(name, g, ref[name], ref["abs"][name])
        out[name] = (kind, err)
    print({n: f"{k} {e:.2e}" for n, (k, e) in out.items()}, flush=True)
    bad = {n: v for n, v in out.items() if not summed_ok(v[0], v[1], tol)}
    assert not bad, bad
    return out


def oracle_summed(ref: dict, mlps=("dphi_k", "dphi_v"), weights=("w1", "b1", "w2", "b2")) -> dict:
    """Flatten the oracle backward's summed gradients and their term magnitudes into the
    {name: array, "abs": {name: array}} form check_summed takes."""
    flat = {"dgate": ref["dgate"], "abs": {"dgate": ref["abs"]["dgate"]}}
    for m in mlps:
        for w in weights:
            flat[f"{m}.{w}"] = ref[m][w]
            flat["abs"][f"{m}.{w}"] = ref["abs"][m][w]
    return flat
