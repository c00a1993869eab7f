"""Helpers shared by the GPU parity tests: move seeded inputs to the GPU, run the
HIP path through the binding, and check it against the fp64 oracle with the
acceptance rules (index sets exact except among keys tied within 1e-5 relative of
the k-th score; outputs within 2e-2 (bf16) / 1e-5 (fp32) of the oracle evaluated on
the GPU's own selected set, per row in the max norm)."""
from __future__ import annotations

import numpy as np
import torch

import paper_2106_06899_amd as tk
from oracle import topk_oracle as o
from paper_2106_06899_amd import workloads as wl

RTOL = {wl.F32: 1e-5, wl.BF16: 2e-2}
GRAD_KAPPA = {wl.F32: 1.0, wl.BF16: 1e-3}


def to_dev(t: wl.Tensor, device="cuda"):
    if t.dtype == wl.BF16:
        return torch.from_numpy(np.ascontiguousarray(t.bits)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(t.values)).to(device)


def run_attn(w: wl.Workload, x: dict, chunk=None, debug=True):
    q, k, v = (to_dev(x[n]) for n in ("Q", "K", "V"))
    res = tk.attn(q, k, v, w.k, w.chunk if chunk is None else chunk, w.causal, w.scale, debug=debug)
    torch.cuda.synchronize()
    return res


def run_ffn(w: wl.Workload, x: dict, chunk=None, debug=True):
    a, b, c = (to_dev(x[n]) for n in ("X", "W1", "W2"))
    res = tk.ffn(a, b, c, w.k, w.chunk if chunk is None else chunk, debug=debug)
    torch.cuda.synchronize()
    return res


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def check_attn(w: wl.Workload, x: dict, out, idx, rows=None, report=None):
    """Check GPU results for `rows` ([R, 3] of (b, h, i); default: all rows)."""
    Q, K, V = (x[n].values for n in ("Q", "K", "V"))
    if rows is None:
        B, H, L = w.B, w.H, w.Lq
        rows = np.stack(np.meshgrid(np.arange(B), np.arange(H), np.arange(L), indexing="ij"), -1).reshape(-1, 3)
    rows = np.asarray(rows)
    ref = o.oracle_attn_rows(Q, K, V, w.k, w.causal, w.scale, rows)
    g_idx = idx.cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]].astype(np.int64)
    g_out = _f64(out)[rows[:, 0], rows[:, 1], rows[:, 2]]
    Qr = Q[rows[:, 0], rows[:, 1], rows[:, 2]]

    def scores_of(r, js):
        b, h, _ = rows[r]
        return Qr[r].astype(np.float64) @ K[b, h][js].astype(np.float64).T

    def valid_of(r, js):
        _, _, i = rows[r]
        lim = min(i + 1, w.Lk) if w.causal else w.Lk
        return (js >= 0) & (js < lim)

    n_bad, n_tie, first = o.check_index_sets(g_idx, ref["idx"], ref["sigma_k"], ref["sigma_k1"], ref["k_eff"],
                                             scores_of, valid_of)
    assert n_bad == 0, f"{n_bad} rows with a wrong index set; first row {rows[first].tolist()}: " \
                       f"gpu {sorted(g_idx[first][g_idx[first] >= 0].tolist())[:12]} " \
                       f"oracle {sorted(ref['idx'][first][ref['idx'][first] >= 0].tolist())[:12]}"
    # outputs vs the oracle evaluated on the GPU's own (validated) index set
    ref_out = np.empty_like(g_out)
    w_ref = np.empty(g_idx.shape)
    for (b, h) in sorted({(int(r[0]), int(r[1])) for r in rows}):
        sel = np.nonzero((rows[:, 0] == b) & (rows[:, 1] == h))[0]
        ref_out[sel], w_ref[sel] = o.from_indices(Qr[sel], K[b, h], V[b, h], g_idx[sel], "softmax", w.scale)
    ratio = o.output_rel_errors(g_out, ref_out, w_ref, float(np.abs(V).max()))
    rtol = RTOL[w.dtype]
    assert np.all(ratio <= rtol), f"output error {ratio.max():.3e} > {rtol} at row {rows[int(np.argmax(ratio))].tolist()}"
    if report is not None:
        report.update(rows=len(rows), tie_rows=int(n_tie), max_err=float(ratio.max()))
    return ratio


def check_ffn(w: wl.Workload, x: dict, out, idx, rows=None, report=None):
    X, W1, W2 = (x[n].values for n in ("X", "W1", "W2"))
    rows = np.arange(w.N) if rows is None else np.asarray(rows)
    ref = o.oracle_ffn_rows(X, W1, W2, w.k, rows)
    g_idx = idx.cpu().numpy()[rows].astype(np.int64)
    g_out = _f64(out)[rows]
    Xr = X[rows].astype(np.float64)

    def scores_of(r, js):
        return Xr[r] @ W1[js].astype(np.float64).T

    def valid_of(r, js):
        return (js >= 0) & (js < w.d_ff)

    n_bad, n_tie, first = o.check_index_sets(g_idx, ref["idx"], ref["sigma_k"], ref["sigma_k1"], ref["k_eff"],
                                             scores_of, valid_of)
    assert n_bad == 0, f"{n_bad} rows with a wrong index set; first row {int(rows[first])}"
    ref_out, w_ref = o.from_indices(Xr, W1, W2, g_idx, "relu")
    ratio = o.output_rel_errors(g_out, ref_out, w_ref, float(np.abs(W2).max()))
    rtol = RTOL[w.dtype]
    assert np.all(ratio <= rtol), f"output error {ratio.max():.3e} > {rtol} at row {int(rows[int(np.argmax(ratio))])}"
    if report is not None:
        report.update(rows=len(rows), tie_rows=int(n_tie), max_err=float(ratio.max()))
    return ratio


def sample_attn_rows(w: wl.Workload, n: int, seed=0):
    """Rows spread over heads, chunk boundaries, the first and last rows and (causal) rows < k."""
    rng = np.random.Generator(np.random.PCG64(seed))
    picks = set()
    C = w.chunk or w.Lq
    for b in range(w.B):
        for h in range(w.H):
            for i in (0, 1, w.Lq - 1, min(C, w.Lq - 1), min(C - 1, w.Lq - 1), min(w.k - 1, w.Lq - 1)):
                picks.add((b, h, i))
    picks = sorted(picks)
    rng.shuffle(picks)
    picks = picks[: n // 2]
    rest = n - len(picks)
    rand = np.stack([rng.integers(0, w.B, rest), rng.integers(0, w.H, rest), rng.integers(0, w.Lq, rest)], -1)
    return np.concatenate([np.array(picks, dtype=np.int64).reshape(-1, 3), rand]).astype(np.int64)


def grad_out(shape, dtype, seed) -> wl.Tensor:
    """A seeded standard-normal output gradient in the workload's dtype."""
    rng = np.random.Generator(np.random.PCG64(seed))
    g = rng.standard_normal(shape).astype(np.float32)
    if dtype == wl.BF16:
        bits = wl.f32_to_bf16_bits(g)
        return wl.Tensor(wl.bf16_bits_to_f32(bits), bits, wl.BF16)
    return wl.Tensor(g, None, wl.F32)


def check_grad_rows(name, got, ref, mag, dtype):
    """Backward acceptance rule, per row (per key for d_K, d_V): max_t |g - r| <= rtol *
    max(max_t |r|, kappa * max_t a), where a is the row's sum of absolute terms from the
    oracle (the scale of rounding in a sum of terms of mixed signs), rtol = 2e-2 (bf16)
    / 1e-5 (fp32), kappa = 1e-3 (bf16) / 1 (fp32); plus the tensor-wide rule (error
    over the largest reference entry). Returns the largest per-row ratio. got: GPU
    gradient (tensor or array); ref, mag: the oracle's gradient and magnitudes."""
    g = np.asarray(got.float().cpu().numpy() if hasattr(got, "cpu") else got, dtype=np.float64)
    g = g.reshape(-1, g.shape[-1])
    r = ref.reshape(-1, ref.shape[-1])
    a = mag.reshape(-1, mag.shape[-1])
    rtol = RTOL[dtype]
    err = np.abs(g - r).max(axis=1)
    own = np.maximum(np.abs(r).max(axis=1), GRAD_KAPPA[dtype] * a.max(axis=1))
    zero = own == 0
    assert not np.any(err[zero]), f"{name}: non-zero gradient where every term is zero"
    ratio = np.where(zero, 0.0, err / np.where(zero, 1.0, own))
    assert np.all(ratio <= rtol), f"{name}: error {ratio.max():.3e} > {rtol} at row {int(np.argmax(ratio))}"
    whole = err.max() / max(float(np.abs(r).max()), 1e-30)
    assert whole <= rtol, f"{name}: tensor-wide error {whole:.3e} > {rtol}"
    return float(ratio.max())
