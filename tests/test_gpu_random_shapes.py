"""Seeded random shapes through every compute entry point, against the fp64
oracle.

The shapes are drawn once, at import, from a fixed seed: dimensions are
log-uniform multiples of 32 (32 .. 16384 for m and n, 32 .. 8192 for r),
decode batches uniform in 1 .. 16, and prefill / training token counts
log-uniform in 1 .. 700, so most cases are small and a few reach several
thousand rows.  The draws land on plan boundaries that the hand-picked
cases do not name: odd word counts, single-row-group layers, ranks far
above or below the layer dimensions, slab splits with a short last slab.

Each case prints its shape before it touches the GPU.  Bars are those of
the named-shape tests: decode outputs element-wise within
2^-7 |ref| + 1e-3 rms(ref) and per-row relative L2 5e-3; prefill outputs
within 2^-6 |ref| + 6e-3 rms(ref) (two fp16 operand roundings) and 5e-3;
training dx within relative L2 5e-3 per token and each scale gradient
within the larger of 1e-3 relative and four times the error predicted by a
first-order model of the path's fp16 roundings (tests/rounding_model.py,
calibrated on the CPU; at short contractions the roundings alone reach
1e-3).  Where the decode workspace fits the
library's own array, the allocation-free entry point must give the same
bits as af1_linear_gemv."""
import numpy as np
import pytest
import torch

from paper_2609_06161_amd import af1, synth
from paper_2609_06161_amd.layer import (DeviceLayer, LayerStream, bf16_bits_to_f64,
                                        gemv_multi, to_device)
from rounding_model import rounding_noise

pytestmark = pytest.mark.gpu

TOL = 5e-3
GRAD_TOL = 1e-3


def _draw_cases(seed=20261202):
    rng = np.random.default_rng(seed)

    def dim(lo, hi):
        return int(32 * np.round(np.exp(rng.uniform(np.log(lo / 32), np.log(hi / 32)))))

    def tokens(hi=700):
        return max(1, int(np.exp(rng.uniform(0.0, np.log(hi)))))

    cases = []
    for kind, count in (("gemv", 40), ("gemm", 24), ("multi", 16), ("stream", 16),
                        ("train", 16)):
        for _ in range(count):
            c = {"kind": kind, "seed": int(rng.integers(1 << 30))}
            if kind == "gemv":
                c.update(m=dim(32, 16384), n=dim(32, 16384), r=dim(32, 8192),
                         b=int(rng.integers(1, 17)), outliers=bool(rng.integers(2)))
            elif kind in ("gemm", "train"):
                # training dims bounded for the error model's dense m x n product
                hi = (16384, 4096) if kind == "gemm" else (4096, 2048)
                c.update(m=dim(32, hi[0]), n=dim(32, hi[0]), r=dim(32, hi[1]), T=tokens())
                # keep the oracle's T x (m + n) x r work to a few seconds
                while c["T"] > 1 and c["T"] * c["r"] * (c["m"] + c["n"]) > 4e9:
                    c["T"] //= 2
            elif kind == "multi":
                c.update(n=dim(32, 16384), b=int(rng.integers(1, 17)),
                         layers=[(dim(32, 8192), dim(32, 4096))
                                 for _ in range(int(rng.integers(2, 5)))])
            else:
                items, prev_m = [], None
                for _ in range(int(rng.integers(1, 6))):
                    wait = prev_m is not None and bool(rng.integers(2))
                    m = dim(32, 8192)
                    items.append((m, prev_m if wait else dim(32, 8192), dim(32, 4096), wait))
                    prev_m = m
                c.update(b=int(rng.integers(1, 17)), items=items)
            cases.append(c)
    return cases


CASES = _draw_cases()


def _case_id(c):
    if c["kind"] in ("gemv",):
        return f"gemv-{c['m']}x{c['n']}-r{c['r']}-b{c['b']}"
    if c["kind"] in ("gemm", "train"):
        return f"{c['kind']}-{c['m']}x{c['n']}-r{c['r']}-T{c['T']}"
    if c["kind"] == "multi":
        return f"multi-n{c['n']}-b{c['b']}-" + "-".join(f"{m}r{r}" for m, r in c["layers"])
    return f"stream-b{c['b']}-" + "-".join(f"{m}x{n}r{r}{'w' if w else ''}"
                                           for m, n, r, w in c["items"])


def max_row_rel_l2(y, ref):
    worst = 0.0
    for a, e in zip(np.asarray(y, np.float64), np.asarray(ref, np.float64)):
        ne = np.linalg.norm(e)
        worst = max(worst, np.linalg.norm(a - e) / ne if ne > 0 else float(np.abs(a).max()))
    return worst


def elementwise_ok(y, ref, rel, abs_rms):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    bad = ~(np.abs(y - ref) <= rel * np.abs(ref) + abs_rms * scale)
    return not bad.any(), np.argwhere(bad)[:5]


def oracle_y(oracle, lin, x):
    return oracle.forward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid,
                          lin.s_in, x)


def nan_out(rows, m):
    return torch.full((rows, m), 0x7FC0, dtype=torch.int16, device="cuda")


def check_decode(got, ref, what):
    ok, where = elementwise_ok(got, ref, 2 ** -7, 1e-3)
    err = max_row_rel_l2(got, ref)
    assert err <= TOL and ok, (what, err, where)


def run_gemv(oracle, c):
    lin = synth.make_linear(c["seed"], c["m"], c["n"], c["r"], c["b"], outliers=c["outliers"])
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    y = nan_out(c["b"], c["m"])
    L.gemv(x, y=y)
    torch.cuda.synchronize()
    check_decode(bf16_bits_to_f64(y), oracle_y(oracle, lin, lin.x), "gemv")
    if af1.af1_gemv_workspace_bytes(c["m"], c["n"], c["r"], c["b"]) <= af1.AF1_GEMV_SCRATCH_BYTES:
        y0 = nan_out(c["b"], c["m"])
        af1.af1_linear_gemv_noalloc(L.desc, x, c["b"], y0)
        torch.cuda.synchronize()
        assert torch.equal(y0, y)


def run_gemm(oracle, c):
    lin = synth.make_linear(c["seed"], c["m"], c["n"], c["r"], c["T"])
    L = DeviceLayer.from_host(lin)
    y = nan_out(c["T"], c["m"])
    L.gemm(to_device(lin.x), y=y)
    torch.cuda.synchronize()
    got, ref = bf16_bits_to_f64(y), oracle_y(oracle, lin, lin.x)
    ok, where = elementwise_ok(got, ref, 2 ** -6, 6e-3)
    err = max_row_rel_l2(got, ref)
    assert err <= TOL and ok, (err, where)


def run_multi(oracle, c):
    b, n = c["b"], c["n"]
    x = synth.make_activations(c["seed"], b, n)
    lins = []
    for i, (m, r) in enumerate(c["layers"]):
        lin = synth.make_linear(c["seed"] + i + 1, m, n, r, b)
        lin.x = x
        lins.append(lin)
    layers = [DeviceLayer.from_host(lin) for lin in lins]
    ys = [nan_out(b, lin.m) for lin in lins]
    gemv_multi(layers, to_device(x), ys=ys)
    torch.cuda.synchronize()
    for k, (lin, y) in enumerate(zip(lins, ys)):
        check_decode(bf16_bits_to_f64(y), oracle_y(oracle, lin, x), ("layer", k))


def run_stream(oracle, c):
    b = c["b"]
    lins, entries, prev = [], [], None
    for i, (m, n, r, wait) in enumerate(c["items"]):
        lin = synth.make_linear(c["seed"] + 7 * i, m, n, r, b)
        x = prev if wait else to_device(lin.x)
        y = nan_out(b, m)
        entries.append((DeviceLayer.from_host(lin), x, y, wait))
        lins.append(lin)
        prev = y
    S = LayerStream(entries, b)
    S.run()
    torch.cuda.synchronize()
    assert S.error_word() == 0
    for k, ((_, x, y, _), lin) in enumerate(zip(entries, lins)):
        xin = x.detach().cpu().numpy().view(np.uint16)
        check_decode(bf16_bits_to_f64(y), oracle_y(oracle, lin, xin), ("item", k))


def run_train(oracle, c):
    lin = synth.make_linear(c["seed"], c["m"], c["n"], c["r"], c["T"])
    dy = synth.make_output_grad(c["seed"] + 1, c["T"], c["m"])
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    y, saved = L.forward_train(x)
    dx, grads = L.backward(x, to_device(dy), saved)
    y_inf = L.gemm(x)
    torch.cuda.synchronize()
    assert torch.equal(y, y_inf)
    rdx, rout, rmid, rin = oracle.backward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out,
                                           lin.s_mid, lin.s_in, lin.x, dy)
    e = max_row_rel_l2(bf16_bits_to_f64(dx), rdx)
    assert e <= TOL, e
    noise = rounding_noise(oracle, lin, dy)
    for name, t, ref, sigma in zip(("ds_out", "ds_mid", "ds_in"), grads, (rout, rmid, rin), noise):
        err = float(np.linalg.norm(t.detach().cpu().numpy().astype(np.float64) - ref))
        assert err <= max(GRAD_TOL * np.linalg.norm(ref), 4 * sigma), (name, err, sigma)


RUNNERS = {"gemv": run_gemv, "gemm": run_gemm, "multi": run_multi, "stream": run_stream,
           "train": run_train}


@pytest.mark.parametrize("case", CASES, ids=[_case_id(c) for c in CASES])
def test_random_shape(oracle, case):
    print(f"random case {_case_id(case)} seed={case['seed']}", flush=True)
    RUNNERS[case["kind"]](oracle, case)
