"""Latency predictor of LPRS (Sec. 3.2.1), trained on the measured attention step.

LPRS picks, for a pending prefill request, the chunk size whose predicted
batch latency is closest to a target T* under an asymmetric penalty.  The
predictor maps the 16 features of a candidate batch (Table 1's 11 raw
statistics, Table 2's 5 derived ones) to its latency; here that latency is
the one of this library's attention step (cp_kv_append + cp_attn_mixed) on
one MI355X, measured by ``bench.py --latency-table`` or by the closed-loop
serving run of ``bench.py --sched``.

* :class:`LatencyPredictor` - the MLP of Table 7: hidden layers (128, 64, 32),
  ReLU, dropout 0.1, AdamW (lr 2e-3, weight decay 1e-3), 300 epochs,
  mini-batch 256, on the weighted asymmetric Huber loss of Eq. 5.  Training
  runs in torch on the CPU; online inference runs in the C++ scheduler
  (``load_into``), which also builds the features and runs Algorithm 1.
* :func:`accuracy` - MAE, RMSE, MAPE (Eq. 15–17) and Table 8's error
  percentiles and bounded-error ratios.

Constants the paper leaves open (Huber threshold, asymmetry factor, number
of buckets) are module defaults.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .sched import FEATURES, NUM_FEATURES, batch_features  # noqa: F401  (C++ feature builder)

RAW_FEATURES = FEATURES[:11]

HUBER_DELTA = 0.25      # in units of the target scale (the training set's median latency)
UNDER_WEIGHT = 2.0      # factor on underestimated samples (prediction below the measurement)
N_BUCKETS = 8           # scheduled-token buckets of the sample weights


def table_features(columns: dict) -> np.ndarray:
    """Feature matrix [n, 16] (cp_sched.h order) from a latency table's
    columns (name -> array).  The derived features are formed from the raw
    ones as Table 2 defines them; memory columns a table lacks are zero."""
    n = len(next(iter(columns.values())))
    raw = {k: np.asarray(columns[k], dtype=np.float64) if k in columns else np.zeros(n)
           for k in RAW_FEATURES}
    dec, pf = raw["decode_tokens"], raw["prefill_tokens"]
    avg = raw["sum_decode_context_len"] / np.maximum(dec, 1.0)
    raw.update(bias=np.ones(n), scheduled_tokens=dec + pf, avg_decode_ctx=avg,
               decode_ctx_interaction=dec * avg,
               prefill_interaction=pf * raw["prefill_processed_tokens"])
    return np.stack([raw[k] for k in FEATURES], axis=1)


def downsample(X, y, cap=3000, seed=0):
    """Caps over-represented batch shapes (Sec. 3.2.1's downsampling): samples
    are grouped by the power-of-two bucket of their scheduled tokens and by
    whether the batch holds prefill work, and each group keeps at most
    ``cap`` samples drawn at random.  Returns the kept indices, sorted."""
    X = np.asarray(X, dtype=np.float64)
    st = X[:, FEATURES.index("scheduled_tokens")]
    has_pf = X[:, FEATURES.index("prefill_tokens")] > 0
    group = np.floor(np.log2(np.maximum(st, 1.0))).astype(np.int64) * 2 + has_pf
    rng = np.random.default_rng(seed)
    keep = []
    for g in np.unique(group):
        idx = np.flatnonzero(group == g)
        if len(idx) > cap:
            idx = rng.choice(idx, cap, replace=False)
        keep.append(idx)
    return np.sort(np.concatenate(keep))


def split_811(n: int, seed: int = 0):
    """Random 8:1:1 train / validation / test index split (Sec. 4.1)."""
    p = np.random.default_rng(seed).permutation(n)
    a, b = int(round(0.8 * n)), int(round(0.9 * n))
    return p[:a], p[a:b], p[b:]


def accuracy(y, y_hat) -> dict:
    """MAE, RMSE, MAPE (Eq. 15–17) and the absolute-error percentiles and
    bounded-error ratios of Table 8, in the units of y (bounds: 5 % and 10 %
    of the median latency, the relative form of the paper's 5 ms and 10 ms at
    its ~100 ms rounds)."""
    y = np.asarray(y, np.float64)
    e = np.asarray(y_hat, np.float64) - y
    a = np.abs(e)
    med = float(np.median(y))
    p = np.percentile(a, [50, 90, 95, 99])
    return {"n": int(len(y)), "mae": float(a.mean()), "rmse": float(np.sqrt((e * e).mean())),
            "mape_pct": float(100.0 * (a / y).mean()), "p50": float(p[0]), "p90": float(p[1]),
            "p95": float(p[2]), "p99": float(p[3]), "median_latency": med,
            "within_5pct_of_median": float((a <= 0.05 * med).mean()),
            "within_10pct_of_median": float((a <= 0.10 * med).mean()),
            "underestimated": float((e < 0).mean())}


def asymmetric_huber(y, y_hat, delta=HUBER_DELTA, under=UNDER_WEIGHT):
    """Per-sample loss l_i of Eq. 5: Huber on e = y_hat - y (quadratic within
    delta, linear beyond), times ``under`` where the latency is underestimated
    (e < 0)."""
    import torch
    e = y_hat - y
    a = e.abs()
    h = torch.where(a <= delta, 0.5 * e * e, delta * (a - 0.5 * delta))
    return torch.where(e < 0, under * h, h)


def bucket_weights(scheduled_tokens, n_buckets=N_BUCKETS) -> np.ndarray:
    """Bucket-aware sample weights w_i: samples are bucketed by total
    scheduled tokens (quantile edges) and every bucket carries the same total
    weight; weights have mean 1."""
    st = np.asarray(scheduled_tokens, dtype=np.float64)
    edges = np.unique(np.quantile(st, np.linspace(0, 1, n_buckets + 1)[1:-1]))
    b = np.searchsorted(edges, st, side="right")
    counts = np.bincount(b, minlength=len(edges) + 1).astype(np.float64)
    w = 1.0 / counts[b]
    return w * (len(w) / w.sum())


@dataclass
class LatencyPredictor:
    """MLP f_theta: features -> step latency (us).  Inputs are standardised
    with the training set's mean and spread (constant features map to 0);
    the target is divided by the training set's median latency."""

    hidden: tuple = (128, 64, 32)
    dropout: float = 0.1
    x_mean: np.ndarray = field(default=None, repr=False)
    x_std: np.ndarray = field(default=None, repr=False)
    y_scale: float = 1.0
    weights: list = field(default=None, repr=False)  # [(W [out, in], b [out]), ...]

    def fit(self, X, y, X_val=None, y_val=None, epochs=300, lr=2e-3, weight_decay=1e-3,
            batch_size=256, seed=0, verbose=False, progress=None):
        """AdamW on the weighted asymmetric Huber loss (Eq. 5); keeps the
        epoch with the lowest validation loss (training loss if no split)."""
        import torch
        torch.manual_seed(seed)
        X = np.asarray(X, dtype=np.float64)
        y = np.asarray(y, dtype=np.float64)
        self.x_mean = X.mean(axis=0)
        sd = X.std(axis=0)
        # A feature constant over the training set (the bias; the memory
        # state when it never changed) carries no information: its
        # standardised input is pinned to 0 so that a later shift in it
        # cannot move the prediction.
        self.x_std = np.where(sd > 0, sd, np.inf)
        self.y_scale = float(np.median(y))
        st = X[:, FEATURES.index("scheduled_tokens")]
        w = bucket_weights(st)
        layers, d_in = [], X.shape[1]
        for h in self.hidden:
            layers += [torch.nn.Linear(d_in, h), torch.nn.ReLU(), torch.nn.Dropout(self.dropout)]
            d_in = h
        layers.append(torch.nn.Linear(d_in, 1))
        net = torch.nn.Sequential(*layers).double()
        opt = torch.optim.AdamW(net.parameters(), lr=lr, weight_decay=weight_decay)
        xt = torch.from_numpy((X - self.x_mean) / self.x_std)
        yt = torch.from_numpy(y / self.y_scale)
        wt = torch.from_numpy(w)
        if X_val is not None:
            xv = torch.from_numpy((np.asarray(X_val, np.float64) - self.x_mean) / self.x_std)
            yv = torch.from_numpy(np.asarray(y_val, np.float64) / self.y_scale)
            wv = torch.from_numpy(bucket_weights(np.asarray(X_val)[:, FEATURES.index("scheduled_tokens")]))
        gen = torch.Generator().manual_seed(seed)
        best, best_state = math.inf, None
        for ep in range(epochs):
            net.train()
            perm = torch.randperm(len(yt), generator=gen)
            for s in range(0, len(perm), batch_size):
                idx = perm[s:s + batch_size]
                loss = (wt[idx] * asymmetric_huber(yt[idx], net(xt[idx]).squeeze(1))).mean()
                opt.zero_grad()
                loss.backward()
                opt.step()
            net.eval()
            with torch.no_grad():
                if X_val is not None:
                    cur = float((wv * asymmetric_huber(yv, net(xv).squeeze(1))).mean())
                else:
                    cur = float((wt * asymmetric_huber(yt, net(xt).squeeze(1))).mean())
            if cur < best:
                best = cur
                best_state = [p.detach().clone() for p in net.parameters()]
            if verbose and ep % 50 == 0:
                print(f"epoch {ep}: loss {cur:.5f}")
            if progress is not None and (ep + 1) % 25 == 0:
                progress(ep + 1, cur)
        if best_state is None:
            raise RuntimeError("predictor training diverged: every epoch's loss was NaN")
        with torch.no_grad():
            for p, b in zip(net.parameters(), best_state):
                p.copy_(b)
        lin = [m for m in net if isinstance(m, torch.nn.Linear)]
        self.weights = [(m.weight.detach().numpy().copy(), m.bias.detach().numpy().copy())
                        for m in lin]
        return self

    def load_into(self, scheduler):
        """Hands the trained weights to a sched.Scheduler (C++ forward pass)."""
        scheduler.set_predictor(self.weights, self.x_mean, self.x_std, self.y_scale)

    def predict(self, X) -> np.ndarray:
        """Predicted latency (us) for each row of X (numpy forward pass, no dropout)."""
        h = (np.asarray(X, dtype=np.float64) - self.x_mean) / self.x_std
        for i, (W, b) in enumerate(self.weights):
            h = h @ W.T + b
            if i + 1 < len(self.weights):
                h = np.maximum(h, 0.0)
        return h[:, 0] * self.y_scale

    __call__ = predict
