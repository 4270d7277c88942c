"""Micro-benchmarks that calibrate the Section 5.2 time models on this GPU.

    python -m paper_2504_03651_amd.calibrate [--out FILE.json] [--reps K]

Times one iteration of the library (``echo_kv_append`` + ``echo_attn_mixed``)
with events on the current stream for:
  * prefill-only batches: one request of l new tokens, no cached context,
    and batches of several chunks (up to 32k new tokens, some after cached
    context), so that the quadratic term is measured where the GPU is full;
  * decode-only batches: n requests with lengths drawn from several shapes
    (uniform, one long row among short ones, equal lengths);
  * mixed batches: one prefill request next to a decode batch, together with
    the two parts alone;
fits ``estimator.Estimator`` on three quarters of the samples of each kind
(seeded split) and reports the relative error on the rest.  Inputs are seeded
synthetic workloads (GQA 32/8, head_dim 128, bf16 by default).
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import workload as W
from .estimator import DecodeModel, Estimator, MixedModel, PrefillModel

# spin before each timed call: long enough to cover the host's planning
GATE_CYCLES = 1_000_000


def _time(w, reps):
    """GPU time of one iteration (KV append + attention), median over reps.
    Each repetition starts behind a short spin on the stream, so the host's
    validation and planning overlap it and the events see device work only."""
    import torch
    from .session import Iteration
    it = Iteration(w)
    for _ in range(2):
        it.append()
        it.attend()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        torch.cuda._sleep(GATE_CYCLES)
        e0.record()
        it.append()
        it.attend()
        e1.record()
    torch.cuda.synchronize()
    return float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))


def _w(rows, cfg, seed):
    return W.build("calib", rows, {}, cfg["hq"], cfg["hkv"], cfg["d"], kv_dtype=cfg["dtype"],
                   seed=seed)


# prefill batches: (number of chunks, new tokens each, cached context each)
PREFILL_BATCHES = [(1, l, 0) for l in (16, 64, 256, 512, 1024, 2048, 3072, 4096, 6144, 8192,
                                       12288, 16384)] + [
    (2, 4096, 0), (4, 2048, 0), (4, 4096, 0), (8, 2048, 0), (8, 4096, 0), (2, 8192, 0),
    (4, 8192, 0), (16, 1024, 0), (16, 2048, 0), (3, 3072, 0), (6, 1536, 0), (12, 1024, 0),
    (1, 2048, 8192), (1, 2048, 16384), (1, 4096, 16384), (2, 4096, 8192), (4, 2048, 4096),
    (4, 4096, 4096), (8, 1024, 8192), (2, 1024, 30000)]


def samples(cfg, reps, log=print):
    rng = np.random.default_rng(cfg.get("seed", 0))
    pre = []
    for k, l, c in PREFILL_BATCHES:
        t = _time(_w([W.RowSpec(W.PREFILL, c, l)] * k, cfg, l + k), reps)
        pre.append(([(l, c)] * k, t))
        log(f"prefill {k} x l={l} after {c}: {t:.4f} ms")
    dec = []
    for n in (16, 64, 256):
        # lengths up to about 300k cached tokens per batch (host draws stay small)
        his = (1024, 4096, 8192) if n <= 64 else (512, 1024, 2048)
        longs = (4096, 16384, 32768) if n <= 64 else (4096, 8192, 16384)
        for shape in range(8):
            if shape < 3:
                L = rng.integers(64, his[shape], size=n)
            elif shape < 6:
                L = rng.integers(64, 1024, size=n)
                L[0] = longs[shape - 3]
            else:
                L = np.full(n, (512, 1024 if n > 64 else 2048)[shape - 6])
            t = _time(_w([W.RowSpec(W.DECODE, int(x), 1) for x in L], cfg, 100 + shape), reps)
            dec.append(([int(x) + 1 for x in L], t))
            log(f"decode n={n} shape={shape} max={L.max()} mean={L.mean():.0f}: {t:.4f} ms")
    mix = []
    for l in (256, 1024, 2048, 4096):
        for n in (16, 64, 256):
            L = rng.integers(256, 4096 if n <= 64 else 2048, size=n)
            prow = [W.RowSpec(W.PREFILL, 0, l)]
            drows = [W.RowSpec(W.DECODE, int(x), 1) for x in L]
            tp = _time(_w(prow, cfg, 7), reps)
            td = _time(_w(drows, cfg, 8), reps)
            tb = _time(_w(prow + drows, cfg, 9), reps)
            mix.append((l, [int(x) + 1 for x in L], tp, td, tb))
            log(f"mixed l={l} n={n}: prefill {tp:.4f} decode {td:.4f} both {tb:.4f} ms")
    return pre, dec, mix


def fit_and_score(pre, dec, mix, cfg, seed=0):
    rng = np.random.default_rng(seed)

    def split(n):
        idx = rng.permutation(n)
        k = max(1, (3 * n) // 4)
        return np.sort(idx[:k]), np.sort(idx[k:])

    pi, po = split(len(pre))
    pm = PrefillModel.fit_chunks([pre[i][0] for i in pi], [pre[i][1] for i in pi])
    # the paper's own reading, one prompt at a time: single prompts only
    single = [i for i in range(len(pre)) if len(pre[i][0]) == 1 and pre[i][0][0][1] == 0]
    si = [i for i in single if i in set(pi.tolist())]
    so = [i for i in single if i not in set(pi.tolist())]
    pm_single = PrefillModel.fit([pre[i][0][0][0] for i in si], [pre[i][1] for i in si])
    # decode: hold out one sample of each batch size and shape group at random
    di, do = split(len(dec))
    dm_paper = DecodeModel.fit([dec[i][0] for i in di], [dec[i][1] for i in di])
    dm = DecodeModel.fit([dec[i][0] for i in di], [dec[i][1] for i in di], intercept=True)
    mi, mo = split(len(mix))
    cols = ([mix[i][2] for i in mi], [mix[i][3] for i in mi], [mix[i][4] for i in mi])
    mm_paper = MixedModel.fit(*cols)
    mm_sum = MixedModel.fit(*cols, form="sum")

    def mixed_err(mm):
        return float(np.mean([abs(float(mm.predict(mix[i][2], mix[i][3])) - mix[i][4]) / mix[i][4]
                              for i in mo]))
    # the estimator keeps the form that predicts the held-out mixed batches better
    mm = mm_sum if mixed_err(mm_sum) < mixed_err(mm_paper) else mm_paper
    est = Estimator(pm, dm, mm, cfg)

    def rel(pred, t):
        return abs(pred - t) / t

    report = {
        "prefill_heldout": [(len(pre[i][0]), pre[i][0][0][0], pre[i][0][0][1], pre[i][1],
                             pm.predict_chunks(pre[i][0])) for i in po],
        "prefill_heldout_single_prompt_fit": [(1, pre[i][0][0][0], 0, pre[i][1],
                                               float(pm_single.predict(pre[i][0][0][0])))
                                              for i in so],
        "decode_heldout_paper_form": [(len(dec[i][0]), int(max(dec[i][0])),
                                       float(np.mean(dec[i][0])), dec[i][1],
                                       dm_paper.predict(dec[i][0])) for i in do],
        "decode_heldout": [(len(dec[i][0]), int(max(dec[i][0])), float(np.mean(dec[i][0])),
                            dec[i][1], dm.predict(dec[i][0])) for i in do],
        "mixed_heldout": [(mix[i][0], len(mix[i][1]), mix[i][4],
                           est.batch_time([mix[i][0]], mix[i][1])) for i in mo],
    }
    errs = {k: float(np.mean([rel(r[-1], r[-2]) for r in v])) for k, v in report.items()}
    errs["mixed_heldout_given_parts_paper_form"] = mixed_err(mm_paper)
    errs["mixed_heldout_given_parts_sum_form"] = mixed_err(mm_sum)
    # the max term's share of the decode time (split-KV should keep it small)
    share = [dm.coef(len(b))[0] * max(b) / dm.predict(b) for b, _ in dec]
    est.config = dict(cfg, decode_paper_form=dm_paper.__dict__, mixed_paper_form=mm_paper.__dict__,
                      prefill_single_prompt_fit=pm_single.__dict__)
    return est, report, errs, float(np.mean(share))


def markdown(out, command):
    """A short summary of a calibration run."""
    c, e = out["coefficients"], out["heldout_mean_rel_error"]
    p, d, m = c["prefill"], c["decode"], c["mixed"]
    lines = [f"# Estimator calibration ({c['config']['hq']}/{c['config']['hkv']} heads, "
             f"head_dim {c['config']['d']}, {c['config']['dtype']})", "",
             "```", command, "```", "",
             "Times are the GPU time of one iteration of the library (KV append + attention; "
             "host planning excluded), median of the repetitions, events on the stream.", "",
             f"* prefill T = max(alpha l^2 + beta l, c): alpha = {p['alpha']:.4g} ms, "
             f"beta = {p['beta']:.4g} ms, c = {p['c']:.4g} ms (fitted on batches of chunks, "
             f"priced as alpha sum(n^2 + 2 n ctx) + beta sum(n)); fitted on single prompts "
             f"only: alpha = {c['config']['prefill_single_prompt_fit']['alpha']:.4g}, beta = "
             f"{c['config']['prefill_single_prompt_fit']['beta']:.4g}, c = "
             f"{c['config']['prefill_single_prompt_fit']['c']:.4g}",
             "* decode T = gamma max(L) + delta mean(L) + eps, per batch size n:", ""]
    lines += ["| n | gamma (ms/token) | delta (ms/token) | eps (ms) |", "|---|---|---|---|"]
    for i, n in enumerate(d["sizes"]):
        lines.append(f"| {n} | {d['gamma'][i]:.4g} | {d['delta'][i]:.4g} | {d['eps'][i]:.4g} |")
    pm = c["config"]["mixed_paper_form"]
    lines += ["", f"* mixed: paper form lam = {pm['lam']:.4g}; sum form kappa = "
              f"{m['kappa']:.4g} ms (used: {m['form']})",
              f"* share of the max(L) term in decode time: {out['decode_max_term_share']:.3f}",
              "", "Held-out mean relative error (a quarter of the samples, seeded split):", "",
              "| model | error |", "|---|---|"]
    for k, v in e.items():
        lines.append(f"| {k} | {v:.3f} |")
    lines += ["", "Samples (ms):", "", "| prefill chunks | new tokens each | cached each | time |",
              "|---|---|---|---|"]
    lines += [f"| {len(b)} | {b[0][0]} | {b[0][1]} | {t:.4f} |" for b, t in out["samples"]["prefill"]]
    lines += ["", "| decode n | max L | mean L | time |", "|---|---|---|---|"]
    lines += [f"| {len(b)} | {max(b)} | {sum(b) / len(b):.0f} | {t:.4f} |"
              for b, t in out["samples"]["decode"]]
    lines += ["", "| mixed l | n | prefill | decode | both |", "|---|---|---|---|---|"]
    lines += [f"| {l} | {len(L)} | {tp:.4f} | {td:.4f} | {tb:.4f} |"
              for l, L, tp, td, tb in out["samples"]["mixed"]]
    return "\n".join(lines) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--out", default=None, help="write the fitted coefficients (JSON)")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--hq", type=int, default=32)
    ap.add_argument("--hkv", type=int, default=8)
    ap.add_argument("--d", type=int, default=128)
    ap.add_argument("--fp8", action="store_true")
    ap.add_argument("--md", default=None, help="write a markdown summary")
    a = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        sys.exit("calibration needs a GPU")
    from . import echo
    echo.lib()
    cfg = dict(hq=a.hq, hkv=a.hkv, d=a.d, dtype=W.KV_FP8 if a.fp8 else W.KV_BF16)
    log = lambda s: print(s, flush=True)
    pre, dec, mix = samples(cfg, a.reps, log)
    est, report, errs, share = fit_and_score(pre, dec, mix, cfg)
    out = {"coefficients": est.to_dict(), "heldout_mean_rel_error": errs,
           "decode_max_term_share": share, "samples": {"prefill": pre, "decode":
           [(b, t) for b, t in dec], "mixed": mix}, "heldout": report}
    log(json.dumps({"coefficients": est.to_dict(), "heldout_mean_rel_error": errs,
                    "decode_max_term_share": share}))
    if a.out:
        with open(a.out, "w") as f:
            json.dump(out, f)
    if a.md:
        cmd = "python -m paper_2504_03651_amd.calibrate " + " ".join(
            argv if argv is not None else sys.argv[1:])
        with open(a.md, "w") as f:
            f.write(markdown(out, cmd))
    return out


if __name__ == "__main__":
    main()
