"""Execution-time and KV-memory estimators of Section 5, fitted to this library.

Section 5.2 models the time of an iteration with three forms whose
coefficients come from micro-benchmarks run before deployment:

  prefill of one request of l tokens    T_p = max(alpha l^2 + beta l, c)
  decode batch with lengths L           T_d = gamma max(L) + delta mean(L)
  batch holding both                    T_b = lam max(T_p, T_d) + (1 - lam) min(T_p, T_d)

and Section 5.3 bounds the KV memory of online requests in the next window by
mu + 2 sigma of the last window's samples.

Here the times are those of one iteration of this library (KV append plus
attention), measured by ``calibrate.py``; the decode form is fitted per batch
size n (its mean term cannot see n) and delta is interpolated linearly in n.
Fitting is plain least squares (NumPy); nothing here touches the GPU.
"""
from __future__ import annotations

from dataclasses import asdict, dataclass, field

import numpy as np


def _nnls(cols, y):
    """Least squares y ~ sum_j a_j cols[j] with every a_j >= 0: the best of the
    unconstrained fits over each subset of the columns whose solution is
    non-negative (a handful of columns, so every subset is tried)."""
    A = np.stack([np.asarray(c, np.float64) for c in cols], 1)
    y = np.asarray(y, np.float64)
    k = A.shape[1]
    best = (float(y @ y), np.zeros(k))
    for mask in range(1, 1 << k):
        j = [i for i in range(k) if mask >> i & 1]
        sol, *_ = np.linalg.lstsq(A[:, j], y, rcond=None)
        if (sol < 0).any():
            continue
        full = np.zeros(k)
        full[j] = sol
        r = float(np.sum((A @ full - y) ** 2))
        if r < best[0]:
            best = (r, full)
    return [float(v) for v in best[1]]


def _nnls2(x1, x2, y):
    return tuple(_nnls([x1, x2], y))


@dataclass
class PrefillModel:
    alpha: float = 0.0
    beta: float = 0.0
    c: float = 0.0

    def predict(self, l):
        l = np.asarray(l, np.float64)
        return np.maximum(self.alpha * l * l + self.beta * l, self.c)

    @classmethod
    def fit(cls, l, t):
        """Chooses c among the measured times (the floor that short prompts
        cannot go below) and fits alpha, beta >= 0 to the points above it;
        keeps the choice with the smallest squared relative error."""
        l = np.asarray(l, np.float64)
        t = np.asarray(t, np.float64)
        best = None
        for c in np.unique(np.concatenate([[0.0], t])):
            m = t > c
            if m.sum() < 2:
                continue
            a, b = _nnls2(l[m] ** 2 / t[m], l[m] / t[m], np.ones(int(m.sum())))
            mdl = cls(a, b, float(c))
            err = float(np.sum(((mdl.predict(l) - t) / t) ** 2))
            if best is None or err < best[0]:
                best = (err, mdl)
        return best[1]


    def predict_chunks(self, chunks):
        """A batch of prefill chunks (n new tokens after ctx cached ones) in
        one launch: the work terms add and the floor applies once (a chunk
        has n ctx + n^2 / 2 (query, key) pairs, priced at 2 alpha each, which
        is alpha l^2 for a whole prompt of l tokens)."""
        work = sum(self.alpha * (n * n + 2.0 * n * c) + self.beta * n for n, c in chunks)
        return max(float(work), self.c)

    @classmethod
    def fit_chunks(cls, batches, t):
        """As fit(), from batches of prefill chunks [(n, ctx), ...] priced by
        predict_chunks: several chunks per batch make alpha identifiable on
        GPUs where one prompt of a few thousand tokens does not fill the
        machine (its time then grows about linearly)."""
        t = np.asarray(t, np.float64)
        q = np.array([sum(n * n + 2.0 * n * c for n, c in b) for b in batches], np.float64)
        l = np.array([sum(n for n, _c in b) for b in batches], np.float64)
        best = None
        for c in np.unique(np.concatenate([[0.0], t])):
            m = t > c
            if m.sum() < 2:
                continue
            a, b = _nnls2(q[m] / t[m], l[m] / t[m], np.ones(int(m.sum())))
            mdl = cls(a, b, float(c))
            pred = np.array([mdl.predict_chunks(x) for x in batches])
            err = float(np.sum(((pred - t) / t) ** 2))
            if best is None or err < best[0]:
                best = (err, mdl)
        return best[1]


@dataclass
class DecodeModel:
    """gamma, delta (and eps) per batch size; coefficients interpolate linearly
    in n.  eps is a constant per iteration: zero in the paper's form; fitted
    with ``intercept=True`` (launches and planning, which dominate small
    batches on this library)."""
    sizes: list = field(default_factory=list)
    gamma: list = field(default_factory=list)
    delta: list = field(default_factory=list)
    eps: list = field(default_factory=list)

    def coef(self, n):
        s = np.asarray(self.sizes, np.float64)
        e = self.eps if self.eps else [0.0] * len(self.sizes)
        return (float(np.interp(n, s, self.gamma)), float(np.interp(n, s, self.delta)),
                float(np.interp(n, s, e)))

    def predict(self, L):
        L = np.asarray(L, np.float64)
        g, d, e = self.coef(len(L))
        return g * float(L.max()) + d * float(L.mean()) + e

    @classmethod
    def fit(cls, batches, t, intercept: bool = False):
        """batches: list of length arrays; t: their times.  One set of
        coefficients >= 0 per distinct batch size, by relative least squares."""
        t = np.asarray(t, np.float64)
        ns = np.array([len(b) for b in batches])
        out = cls()
        for n in sorted(set(ns.tolist())):
            idx = np.nonzero(ns == n)[0]
            mx = np.array([float(np.max(batches[i])) for i in idx])
            mn = np.array([float(np.mean(batches[i])) for i in idx])
            cols = [mx / t[idx], mn / t[idx]] + ([1.0 / t[idx]] if intercept else [])
            sol = _nnls(cols, np.ones(len(idx)))
            out.sizes.append(int(n))
            out.gamma.append(sol[0])
            out.delta.append(sol[1])
            out.eps.append(sol[2] if intercept else 0.0)
        return out


@dataclass
class MixedModel:
    """The paper's form (``form="lambda"``), or ``form="sum"``: T_p + T_d - kappa,
    for an implementation that runs the two kinds of work one after the other
    and shares only the per-iteration overhead kappa (this library does: its
    prefill and decode kernels run back to back on one stream)."""
    lam: float = 1.0
    kappa: float = 0.0
    form: str = "lambda"

    def predict(self, tp, td):
        tp, td = np.asarray(tp, np.float64), np.asarray(td, np.float64)
        if self.form == "sum":
            return tp + td - self.kappa
        return self.lam * np.maximum(tp, td) + (1 - self.lam) * np.minimum(tp, td)

    @classmethod
    def fit(cls, tp, td, tb, form: str = "lambda"):
        """lambda: lam minimising the squared error of tb - min = lam (max - min);
        sum: kappa = mean(tp + td - tb), at least 0."""
        tp, td, tb = (np.asarray(x, np.float64) for x in (tp, td, tb))
        if form == "sum":
            return cls(kappa=max(0.0, float(np.mean(tp + td - tb))), form="sum")
        hi, lo = np.maximum(tp, td), np.minimum(tp, td)
        d = hi - lo
        den = float(d @ d)
        return cls(float(d @ (tb - lo)) / den if den > 0 else 1.0)


@dataclass
class Estimator:
    prefill: PrefillModel
    decode: DecodeModel
    mixed: MixedModel
    config: dict = field(default_factory=dict)

    def batch_time(self, prefill_lens, decode_lens):
        """Estimated iteration time: prefill requests one after another (the
        paper's practice), then combined with the decode batch by lam."""
        tp = float(np.sum(self.prefill.predict(prefill_lens))) if len(prefill_lens) else 0.0
        td = self.decode.predict(decode_lens) if len(decode_lens) else 0.0
        if tp == 0.0 or td == 0.0:
            return tp + td
        return float(self.mixed.predict(tp, td))

    def batch_time_kernel(self, prefill_chunks, decode_lens, decode_unique_tokens=None):
        """The same forms and coefficients read for this library's kernels
        instead of an engine that runs prefills one after another and reads
        every row's KV separately: the prefill chunks of a batch run in one
        launch, so their work terms add and the floor c applies once; a chunk
        of n new tokens after ctx cached ones has n ctx + n^2 / 2 (query, key)
        pairs, which alpha l^2 prices as l^2 / 2 for a whole prompt; decode
        rows that share prefix blocks read them once, so the mean term takes
        the distinct KV tokens per row (decode_unique_tokens / n).
        prefill_chunks: (n, ctx) pairs; decode_lens: the rows' lengths."""
        p = self.prefill
        tp = 0.0
        if len(prefill_chunks):
            work = sum(p.alpha * (n * n + 2.0 * n * c) + p.beta * n for n, c in prefill_chunks)
            tp = max(float(work), p.c)
        td = 0.0
        if len(decode_lens):
            L = np.asarray(decode_lens, np.float64)
            g, d, e = self.decode.coef(len(L))
            mean = float(L.mean()) if decode_unique_tokens is None else decode_unique_tokens / len(L)
            td = g * float(L.max()) + d * mean + e
        if tp == 0.0 or td == 0.0:
            return tp + td
        return float(self.mixed.predict(tp, td))

    def to_dict(self):
        return {"prefill": asdict(self.prefill), "decode": asdict(self.decode),
                "mixed": asdict(self.mixed), "config": self.config}

    @classmethod
    def from_dict(cls, d):
        return cls(PrefillModel(**d["prefill"]), DecodeModel(**d["decode"]),
                   MixedModel(**d["mixed"]), d.get("config", {}))


def kv_memory_bound(samples, k: float = 2.0) -> float:
    """mu + k sigma of the KV memory samples of the last window (Section 5.3:
    a normal model, k = 2 covers about 95% of windows)."""
    x = np.asarray(samples, np.float64)
    return float(x.mean() + k * x.std())
