"""Shared test helpers: move seeded host arrays to the GPU and gate parity."""
import numpy as np

from oracle import favor, metrics

TOL = {"f32": 1e-4, "bf16": 2e-2}


def torch_dtype(name):
    import torch
    return torch.bfloat16 if name == "bf16" else torch.float32


def to_dev(x, dtype="f32"):
    """float32 host array (values exact in dtype) -> contiguous GPU tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(device="cuda", dtype=torch_dtype(dtype)).contiguous()


def to_host(t):
    return t.float().cpu().numpy().astype(np.float64)


def oracle_features(Q, K, W, b, s, kernel=favor.KERNEL_SOFTMAX, kernel_eps=1e-3):
    return (favor.features(Q, W, b, s, kernel, kernel_eps),
            favor.features(K, W, b, s, kernel, kernel_eps))


def parity(out, Q, K, V, W, b, s, causal, dtype, eps=0.0, state_in=None, tol=None,
           heads=None, kernel=favor.KERNEL_SOFTMAX, kernel_eps=1e-3, renormalize=True,
           gate="both", stats=None):
    """Compare a GPU output with the oracle on the same inputs and features.

    heads: optional list of (batch, head) pairs to check (large inputs).
    kernel, kernel_eps, renormalize: the feature kernel and normalisation of the
    call. gate: "both" asserts E_row and E_cond, "cond" only E_cond (regimes
    where D-hat cancels, such as input_scale 1, or cos features at small M:
    E_row has no conditioning term there). Renormalised rows whose denominator
    has no correct bit at the input precision (kappa u >= 1) may be non-finite;
    they are left out. stats: optional dict that receives the per-row condition
    numbers kappa. Returns (E_row, E_cond)."""
    tol = TOL[dtype] if tol is None else tol
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    out = np.asarray(out, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if heads is not None:
        sel = lambda a: np.stack([a[bi, hi] for bi, hi in heads])[:, None]
        Q, K, V, out = sel(Q), sel(K), sel(V), sel(out)
        W = np.stack([W[hi] for _, hi in heads])[:, None]
        b = np.stack([b[hi] for _, hi in heads])[:, None]
        if state_in is not None:
            state_in = sel(np.asarray(state_in, dtype=np.float64))
    Qp, Kp = oracle_features(Q, K, W, b, s, kernel, kernel_eps)
    if causal:
        ref, _ = favor.attn_causal_features(Qp, Kp, V, eps, state_in, renormalize)
    else:
        ref = favor.attn_bidir_features(Qp, Kp, V, eps, renormalize)
    S, den = metrics.error_scale(Qp, Kp, V, causal, state_in=state_in)
    if renormalize:
        # a row whose denominator cancels below the rounding level of its terms
        # (kappa u >= 1, u the unit roundoff of the input dtype) has no correct
        # bit in D-hat: the kernel divides by whatever its sum gave, 0 included,
        # so a non-finite result there is no fault; such rows are left out
        u = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -24
        open_rows = (metrics.kappa(S, den + eps) * u >= 1.0) & ~np.all(np.isfinite(out), axis=-1)
        if open_rows.any():
            out = np.where(open_rows[..., None], ref, out)
    e_row = metrics.err_row(out, ref)
    if not renormalize:
        e_cond = metrics.err_cond_numerator(out, ref, S)
    else:
        e_cond = metrics.err_cond(out, ref, S, den + eps)
    if stats is not None:
        stats["kappa"] = metrics.kappa(S, den + eps)
    if gate == "both":
        assert e_row <= tol, f"E_row {e_row:.3e} > {tol}"
    assert e_cond <= tol, f"E_cond {e_cond:.3e} > {tol}"
    return e_row, e_cond
