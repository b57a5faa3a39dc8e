"""Iteration cost model fitted on this library's kernels (Sec. 4.1).

The paper prices one serving iteration with a latency model per phase,
    t_exec = a0 * Ln + a1 * Ln * La + b,
where Ln is the number of input tokens of the batch's requests and La the
total context they attend to (cached plus input), fitted by least squares on
offline profiles whose sizes step by powers of two; prefill and decode get
separate fits (for prefill La = Ln, nothing being cached yet), and a batch's
time is the sum over its two phases. Checkpointed KV that must come back adds
a swap time linear in the amount moved, and the iteration costs
max(t_exec, t_swap) when the copies overlap execution.

Here the "execution" is the attention step that this library runs, not a
whole model, so besides the paper's form the module fits a second one per
phase whose interaction term is the sum over requests of n_i * a_i (input
tokens times attended tokens of each request). For one request the two forms
coincide; for a batch the paper's Ln * La counts cross-request pairs that no
kernel computes. Both fits are reported.

    python -m paper_2504_09590_amd.costmodel           # profile on the GPU, fit, print JSON
    python -m paper_2504_09590_amd.costmodel --out paper_2504_09590_amd/costmodel_mi355x.json

The profiler builds its batches directly on the device (random bf16 values,
tables from a random permutation of one pool), times each call with HIP
events, and takes the median of its repetitions. costmodel_mi355x.json, next
to this module, holds the model fitted this way on one MI355X; the block
manager's benchmark (manager.main) prices its batches with it.
"""


from __future__ import annotations

import argparse
import json
import os
import sys
from dataclasses import dataclass, field

import numpy as np

FORMS = ("paper", "per_request")


@dataclass
class Sample:
    phase: str          # "prefill" | "decode"
    ln: int             # input tokens of the batch
    la: int             # tokens attended (cached + input), summed over requests
    pairs: int          # sum over requests of n_i * a_i
    t_us: float
    requests: int = 1


def features(form: str, ln, la, pairs) -> np.ndarray:
    ln, la, pairs = (np.asarray(x, dtype=np.float64) for x in (ln, la, pairs))
    if form == "paper":
        inter = ln * la
    elif form == "per_request":
        inter = pairs
    else:
        raise ValueError(f"unknown form {form!r}")
    return np.stack([ln, inter, np.ones_like(ln)], axis=-1)


def _nonneg_lstsq(A: np.ndarray, y: np.ndarray) -> np.ndarray:
    """argmin |A x - y| over x >= 0: every term of the model is a cost (per
    token, per attended pair, per launch), so none may be negative. The
    columns are scaled to unit norm first (they span many decades)."""
    from scipy.optimize import nnls
    norm = np.linalg.norm(A, axis=0)
    norm[norm == 0] = 1.0
    x, _ = nnls(A / norm, y)
    return x / norm


def fit(samples, form: str) -> np.ndarray:
    """(a0, a1, b) >= 0 minimising the squared RELATIVE error over the samples
    (a profile spans several decades of time; plain least squares would fit
    only the largest points)."""
    X = features(form, [s.ln for s in samples], [s.la for s in samples], [s.pairs for s in samples])
    t = np.array([s.t_us for s in samples], dtype=np.float64)
    w = 1.0 / t
    return _nonneg_lstsq(X * w[:, None], t * w)


def fit_swap(sizes_bytes, t_us) -> np.ndarray:
    """(seconds per byte expressed as us/B, fixed us) >= 0 of a linear swap-time model."""
    X = np.stack([np.asarray(sizes_bytes, dtype=np.float64), np.ones(len(sizes_bytes))], axis=-1)
    t = np.asarray(t_us, dtype=np.float64)
    w = 1.0 / t
    return _nonneg_lstsq(X * w[:, None], t * w)


@dataclass
class CostModel:
    coef: dict = field(default_factory=dict)     # (phase, form) -> [a0, a1, b]
    swap: dict = field(default_factory=dict)     # "d2h" / "h2d" -> [us per byte, us]

    def predict(self, phase: str, ln, la, pairs=None, form: str = "paper"):
        a = np.asarray(self.coef[f"{phase}/{form}"], dtype=np.float64)
        if pairs is None:
            pairs = np.asarray(ln) * np.asarray(la)
        return features(form, ln, la, pairs) @ a

    def swap_us(self, nbytes_out: float = 0.0, nbytes_in: float = 0.0) -> float:
        t = 0.0
        for key, n in (("d2h", nbytes_out), ("h2d", nbytes_in)):
            if n > 0:
                g, d = self.swap[key]
                t += g * n + d
        return t

    def iteration_us(self, prefill=None, decode=None, nbytes_out=0.0, nbytes_in=0.0,
                     overlap: bool = False, form: str = "paper") -> float:
        """prefill / decode: (Ln, La, pairs) of each phase's requests, or None."""
        t_exec = 0.0
        for phase, p in (("prefill", prefill), ("decode", decode)):
            if p is not None:
                t_exec += float(self.predict(phase, *p, form=form))
        t_swap = self.swap_us(nbytes_out, nbytes_in)
        return max(t_exec, t_swap) if overlap else t_exec + t_swap

    def to_json(self) -> str:
        return json.dumps({"coef": {k: [float(x) for x in v] for k, v in self.coef.items()},
                           "swap": {k: [float(x) for x in v] for k, v in self.swap.items()}}, indent=1)

    @staticmethod
    def from_json(text: str) -> "CostModel":
        d = json.loads(text)
        return CostModel(coef=d["coef"], swap=d["swap"])


MODEL_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "costmodel_mi355x.json")


def load_fitted(path: str = MODEL_PATH) -> CostModel:
    """The model fitted on one MI355X (written by main with --out)."""
    with open(path) as f:
        return CostModel.from_json(f.read())


def power_grid(lo: int, hi: int) -> list[int]:
    """Powers of two from lo to hi inclusive (the paper's profiling steps)."""
    out, v = [], lo
    while v <= hi:
        out.append(v)
        v *= 2
    return out


def relative_errors(model: CostModel, samples, form: str) -> np.ndarray:
    pred = np.array([float(model.predict(s.phase, s.ln, s.la, s.pairs, form=form)) for s in samples])
    t = np.array([s.t_us for s in samples])
    return np.abs(pred - t) / t


# ---------------------------------------------------------------------------
# profiling on the GPU (this library's kernels)
# ---------------------------------------------------------------------------

class _Pool:
    """One bf16 pool on the device, big enough for the largest profile point."""

    def __init__(self, torch, num_blocks, hkv, d, seed=0):
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        self.k = torch.randn((num_blocks, hkv, 16, d), generator=g, device="cuda").to(torch.bfloat16)
        self.v = torch.randn((num_blocks, hkv, 16, d), generator=g, device="cuda").to(torch.bfloat16)
        self.num_blocks = num_blocks
        self.perm = np.random.default_rng(seed).permutation(num_blocks).astype(np.int32)


def _tables(ctx, pool: _Pool):
    nblk = (np.asarray(ctx) + 15) // 16
    maxb = max(1, int(nblk.max()))
    t = np.full((len(ctx), maxb), -1, dtype=np.int32)
    cur = 0
    for s, n in enumerate(nblk):
        t[s, :n] = pool.perm[cur:cur + n]
        cur += int(n)
    assert cur <= pool.num_blocks
    return t


def _time_us(torch, fn, reps: int) -> float:
    fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b) * 1e3)
    return float(np.median(ts))


def profile_prefill(torch, bros, pool, hq, hkv, d, points, reps=7):
    out = []
    for batch, n in points:
        ctx = np.full(batch, n, dtype=np.int32)           # nothing cached: La = Ln
        tables = torch.from_numpy(_tables(ctx, pool)).cuda()
        cu_q = torch.from_numpy(np.arange(batch + 1, dtype=np.int32) * n).cuda()
        q = torch.randn((batch * n, hq, d), device="cuda").to(torch.bfloat16)
        o = torch.empty_like(q)
        dirs = torch.ones(batch, dtype=torch.int8, device="cuda")
        ctx_d = torch.from_numpy(ctx).cuda()
        t = _time_us(torch, lambda: bros.bros_attn_prefill_chunk(o, q, cu_q, n, pool.k, pool.v, tables, dirs, None,
                                                                 ctx_d, n), reps)
        out.append(Sample("prefill", batch * n, batch * n, batch * n * n, t, batch))
    return out


def profile_decode(torch, bros, pool, hq, hkv, d, points, reps=7):
    out = []
    for batch, c in points:
        ctx = np.full(batch, c, dtype=np.int32)
        tables = torch.from_numpy(_tables(ctx, pool)).cuda()
        q = torch.randn((batch, hq, d), device="cuda").to(torch.bfloat16)
        o = torch.empty_like(q)
        dirs = -torch.ones(batch, dtype=torch.int8, device="cuda")
        ctx_d = torch.from_numpy(ctx).cuda()
        wsb = bros.bros_attn_workspace_size(bros.BROS_WS_DECODE, bros.BROS_BF16, batch, hq, d, c)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        t = _time_us(torch, lambda: bros.bros_attn_decode(o, q, pool.k, pool.v, tables, dirs, None, ctx_d, c,
                                                          workspace=ws), reps)
        out.append(Sample("decode", batch, batch * c, batch * c, t, batch))
    return out


def profile_swap(torch, bros, sizes_bytes, reps=7):
    res = {"d2h": [], "h2d": []}
    top = max(sizes_bytes)
    dev = torch.empty(top, dtype=torch.uint8, device="cuda")
    host = torch.empty(top, dtype=torch.uint8, pin_memory=True)
    for n in sizes_bytes:
        res["d2h"].append(_time_us(torch, lambda: bros.bros_copy_dma(host, dev, n), reps))
        res["h2d"].append(_time_us(torch, lambda: bros.bros_copy_dma(dev, host, n), reps))
    return res


def main(argv=None):
    ap = argparse.ArgumentParser(description="profile this library's kernels and fit the Sec. 4.1 cost model")
    ap.add_argument("--reps", type=int, default=7)
    ap.add_argument("--out", default=None, help="also write the fitted model (CostModel JSON) to this file")
    args = ap.parse_args(argv)
    import torch
    from . import bros
    if not torch.cuda.is_available():
        print("costmodel: no GPU visible", file=sys.stderr)
        sys.exit(1)
    hq, hkv, d = 32, 8, 128                               # Llama-3-8B attention
    fit_pre = [(b, n) for n in power_grid(128, 4096) for b in power_grid(1, 8) if b * n <= 16384]
    fit_dec = [(b, c) for b in power_grid(8, 256) for c in power_grid(256, 8192)]
    held_pre = [(3, 384), (3, 1536), (6, 768), (5, 2048)]
    held_dec = [(48, 768), (96, 3072), (24, 6144), (192, 1536)]
    blocks = max(max(b * c for b, c in fit_dec + held_dec), max(b * n for b, n in fit_pre + held_pre)) // 16 + 16
    pool = _Pool(torch, blocks, hkv, d)
    model = CostModel()
    report = {"shape": {"q_heads": hq, "kv_heads": hkv, "head_dim": d, "dtype": "bf16"}}
    for phase, prof, grid, held in (("prefill", profile_prefill, fit_pre, held_pre),
                                    ("decode", profile_decode, fit_dec, held_dec)):
        fit_s = prof(torch, bros, pool, hq, hkv, d, grid, args.reps)
        held_s = prof(torch, bros, pool, hq, hkv, d, held, args.reps)
        report[phase] = {"fit_points": [vars(s) for s in fit_s], "held_out": [vars(s) for s in held_s]}
        for form in FORMS:
            model.coef[f"{phase}/{form}"] = list(fit(fit_s, form))
            report[phase][form] = {"coef": [float(x) for x in model.coef[f"{phase}/{form}"]],
                                   "max_rel_err_fit": float(relative_errors(model, fit_s, form).max()),
                                   "max_rel_err_held_out": float(relative_errors(model, held_s, form).max())}
    sizes = [16 * m * 2 * hkv * d * 2 for m in power_grid(16, 4096)]   # M blocks' worth of slots, K and V
    sw = profile_swap(torch, bros, sizes, args.reps)
    report["swap"] = {"bytes": sizes, **sw}
    for key in ("d2h", "h2d"):
        model.swap[key] = list(fit_swap(sizes, sw[key]))
        pred = np.array(sizes) * model.swap[key][0] + model.swap[key][1]
        report["swap"][key + "_fit"] = {"us_per_byte": float(model.swap[key][0]), "us": float(model.swap[key][1]),
                                        "GB/s": float(1e-3 / model.swap[key][0]),
                                        "max_rel_err": float(np.max(np.abs(pred - sw[key]) / np.array(sw[key])))}
    report["model"] = json.loads(model.to_json())
    if args.out:
        with open(args.out, "w") as f:
            f.write(model.to_json() + "\n")
    print(json.dumps(report), flush=True)


if __name__ == "__main__":
    main()
