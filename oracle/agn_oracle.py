"""CPU oracle of the Accumulated Gradient Normalization (AGN) hot path.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously
correct statement of what the GPU path computes.  Only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it; the
product path never does.  It shares no code with the HIP library.

What it computes (Hermans, Spanakis, Moeckel, "Accumulated Gradient
Normalization", ACML 2017):

* Algorithm 1 (worker procedure of AGN): a worker pulls the central
  variable, runs lambda local mini-batch SGD steps while accumulating the
  steps in ``a``, divides ``a`` by lambda (the normalization step), commits
  ``a`` and pulls the central variable again.  Without the normalization
  step (``normalize=False``) this is Section 2's DOWNPOUR with accumulated
  gradients; with lambda = 1 both are DOWNPOUR.
* Eq. (1): the committed delta is minus the learning rate times the
  lambda-average of mini-batch mean gradients taken along the local path.
* Eq. (2): the parameter server adds each arriving delta to the central
  variable.
* Section 1 (caption of the asynchronous data-parallelism figure): the
  server applies commits as a FIFO queue; with n homogeneous workers the
  expected staleness of a commit is n - 1.
* Section 4 (the DynSGD comparison): a commit scaled down by its staleness
  (``staleness_scaled=True``), read as the factor 1 / (tau + 1), tau the
  number of commits applied since the worker's last pull.  The paper gives
  only the effect (about 1 / (n - 1) at E[tau] = n - 1); the cited work
  holding the exact rule is not available, so this reading is partly
  unpinned.

Readings of points the paper leaves open (each one is listed in the design
notes of the repository):

* Eq. (1) sums i = 0..lambda, Algorithm 1 runs lambda steps; the oracle
  runs lambda steps.
* One round = every worker runs lambda steps from its last pulled copy;
  then the commits are applied in the given order and each worker pulls
  the central variable right after its own commit.
* Learning rate constant (Section 4: no decay); plain SGD as the local rule.
* Model: ReLU MLP, softmax cross-entropy on the last layer, no activation
  on the output; theta holds all weights and biases; ReLU'(0) = 0.
* Mini-batches: worker k owns rows [k*S, (k+1)*S) with S = floor(N/n);
  local step t (counted over all rounds) uses rows
  k*S + ((t*m + j) mod S), j = 0..m-1.
* Initial weights: He-normal from a SplitMix64 stream (Box-Muller), biases
  zero.
* Precision: tensors are stored in float32 at the points where the GPU
  stores them; every dot product and every reduction is accumulated in
  float64 and rounded to float32 once.  In the bf16 mode the operands of
  every matrix product (inputs, weights, hidden activations after ReLU,
  output-side gradients) are rounded to bfloat16 (round to nearest even)
  first; logits, softmax, bias, updates and commits stay float32, and the
  bias gradient sums the bf16-rounded output-side gradients.
* A float64 storage mode (``dtype=np.float64``) turns every float32
  rounding into the identity; the finite-difference pin uses it.
"""
from __future__ import annotations

import math
from typing import List, Sequence

import numpy as np

__all__ = [
    "splitmix64", "he_normal_init", "bf16_round", "batch_indices",
    "loss_and_grads", "forward", "evaluate", "AGNOracle", "flat_params", "unflat_params", "near_zero_units",
]

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_MIX1 = np.uint64(0xBF58476D1CE4E5B9)
_MIX2 = np.uint64(0x94D049BB133111EB)


# ---------------------------------------------------------------------------
# Initialisation: SplitMix64 (Steele, Lea and Flood, OOPSLA 2014; the
# 64-bit finaliser constants of Vigna's public-domain splitmix64) feeding a
# Box-Muller transform, scaled to He-normal N(0, 2 / d_in).
# ---------------------------------------------------------------------------

def splitmix64(seed: int, first: int, count: int) -> np.ndarray:
    """Outputs number first..first+count-1 of the SplitMix64 stream seeded
    with ``seed``.  Output i is mix(seed + (i + 1) * gamma) mod 2**64."""
    with np.errstate(over="ignore"):
        i = np.arange(first + 1, first + count + 1, dtype=np.uint64)
        z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + i * _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _MIX1
        z = (z ^ (z >> np.uint64(27))) * _MIX2
        z = z ^ (z >> np.uint64(31))
    return z


def he_normal_init(dims: Sequence[int], seed: int, dtype=np.float32):
    """Initial parameters [(W_0, b_0), (W_1, b_1), ...].

    W_l has shape (d_{l+1}, d_l).  Weights are numbered 0, 1, 2, ... in the
    packed order W_0 (row-major), W_1, ...; weight w uses stream outputs 2w
    (u1 = ((x >> 11) + 1) / 2**53, in (0, 1]) and 2w + 1
    (u2 = (x >> 11) / 2**53, in [0, 1)) and takes the value
    sqrt(-2 ln u1) * cos(2 pi u2) * sqrt(2 / d_l), evaluated in float64 and
    rounded once.  Biases start at zero.
    """
    params = []
    w = 0
    for l in range(len(dims) - 1):
        fan_in, fan_out = dims[l], dims[l + 1]
        cnt = fan_in * fan_out
        x = splitmix64(seed, 2 * w, 2 * cnt)
        u1 = ((x[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * 2.0 ** -53
        u2 = (x[1::2] >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
        z = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)
        W = (z * math.sqrt(2.0 / fan_in)).astype(dtype).reshape(fan_out, fan_in)
        params.append((W, np.zeros(fan_out, dtype=dtype)))
        w += cnt
    return params


# ---------------------------------------------------------------------------
# Rounding helpers
# ---------------------------------------------------------------------------

def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); the
    result is returned as float32 holding bf16-representable values."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).reshape(np.shape(x))


class _Prec:
    """Where values are stored: float32 (the GPU's storage) or float64."""

    def __init__(self, dtype, bf16: bool):
        self.dtype = np.dtype(dtype)
        self.bf16 = bf16
        if bf16 and self.dtype != np.float32:
            raise ValueError("bf16 mode stores float32 masters")

    def st(self, x):
        """Store: round a float64 intermediate to the storage type."""
        return np.asarray(x).astype(self.dtype)

    def op(self, x):
        """Operand of a matrix product (bf16-rounded in bf16 mode)."""
        return bf16_round(x) if self.bf16 else x

    @staticmethod
    def mm(a, b):
        """Matrix product accumulated in float64."""
        return np.asarray(a, dtype=np.float64) @ np.asarray(b, dtype=np.float64)


# ---------------------------------------------------------------------------
# FetchNextMiniBatch (Algorithm 1) under the contiguous-shard reading
# ---------------------------------------------------------------------------

def batch_indices(k: int, t: int, m: int, S: int) -> np.ndarray:
    """Row indices of worker k's mini-batch at its local step t.

    Worker k owns the contiguous shard [k*S, (k+1)*S) (Section 1: n shards;
    Section 4: data equally distributed over the n workers) and walks it
    cyclically, m rows per step."""
    j = np.arange(m, dtype=np.int64)
    return np.int64(k) * np.int64(S) + (np.int64(t) * np.int64(m) + j) % np.int64(S)


# ---------------------------------------------------------------------------
# Mini-batch loss and gradient of the ReLU MLP (the gradient term of Eq. 1)
# ---------------------------------------------------------------------------

def forward(params, xb: np.ndarray, prec: _Prec):
    """Forward pass of the ReLU MLP over the rows of xb.

    Returns (H, logits): H[0] is the input batch, H[l+1] =
    relu(H[l] W_l^T + b_l) for the hidden layers (bf16-rounded in bf16
    mode, as operands of the next product), and the stored logits
    H[L-1] W_{L-1}^T + b_{L-1}."""
    L = len(params)
    H = [prec.op(np.asarray(xb, dtype=prec.dtype))]
    for l in range(L - 1):
        W, b = params[l]
        z = prec.st(prec.mm(H[l], prec.op(W).T) + b)
        H.append(prec.op(np.maximum(z, 0)))
    W, b = params[L - 1]
    logits = prec.st(prec.mm(H[L - 1], prec.op(W).T) + b)
    return H, logits


def loss_and_grads(params, xb: np.ndarray, yb: np.ndarray, prec: _Prec):
    """Mean softmax cross-entropy over the m rows of the batch and its
    gradient with respect to every W_l and b_l (Eq. 1: the inner average
    over j = 0..m-1 of per-sample gradients).

    Returns (loss as float64, [(dW_0, db_0), ...])."""
    L = len(params)
    m = xb.shape[0]
    H, logits = forward(params, xb, prec)

    # softmax cross-entropy, evaluated in float64 from the stored logits
    z = logits.astype(np.float64)
    zmax = z.max(axis=1, keepdims=True)
    ez = np.exp(z - zmax)
    s = ez.sum(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(s[:, 0])
    rows = np.arange(m)
    loss = float(np.mean(lse - z[rows, yb]))
    p = ez / s
    onehot = np.zeros_like(p)
    onehot[rows, yb] = 1.0
    dz = prec.st((p - onehot) / m)          # d(mean loss)/d(logits)

    grads = [None] * L
    for l in range(L - 1, -1, -1):
        dzq = prec.op(dz)
        dW = prec.st(prec.mm(dzq.T, H[l]))
        db = prec.st(np.sum(np.asarray(dzq, dtype=np.float64), axis=0))
        grads[l] = (dW, db)
        if l >= 1:
            back = prec.st(prec.mm(dzq, prec.op(params[l][0])))
            dz = back * (H[l] > 0)           # ReLU'(0) = 0
    return loss, grads


def near_zero_units(params, xb: np.ndarray, prec: _Prec, rel: float = 1e-6):
    """Diagnostic for the parity tests, not part of the method: per hidden
    layer (H_1 .. H_{L-1}) the units whose pre-activation, for some row of
    the batch, lies within rel times the sum of the magnitudes of its terms
    of zero.  There a float32 sum taken in another order can land on the
    other side of zero and flip the ReLU derivative (a step at zero), which
    changes that unit's row of the layer's weight gradient and its bias
    gradient by one sample's whole contribution.  The forward pass is the
    one ``forward`` computes."""
    L = len(params)
    H = prec.op(np.asarray(xb, dtype=prec.dtype))
    out = []
    for l in range(L - 1):
        W, b = params[l]
        Wo = prec.op(W)
        z = prec.mm(H, Wo.T) + b
        scale = prec.mm(np.abs(H), np.abs(Wo).T) + np.abs(np.asarray(b, dtype=np.float64))
        out.append(np.flatnonzero((np.abs(z) <= rel * scale).any(axis=0)))
        H = prec.op(np.maximum(prec.st(z), 0))
    return out


# ---------------------------------------------------------------------------
# Evaluation of a model over a labelled set (Section 4: the training and
# validation accuracy of the central variable, the f(t) of Eq. 4)
# ---------------------------------------------------------------------------

def evaluate(params, X: np.ndarray, y: np.ndarray, bf16: bool = False, dtype=np.float32):
    """Per-row softmax cross-entropy and predicted class of the model
    ``params`` on every row of (X, y).

    The logits are those of ``forward`` (stored in the storage type); the
    loss of row j is logsumexp(z_j) - z_{j,y_j}, evaluated in float64 from
    them; the prediction is the index of the largest logit, the lowest such
    index when several are equal.  Returns (row_loss float64 [N],
    pred int64 [N], logits [N][C])."""
    prec = _Prec(dtype, bf16)
    X = np.asarray(X)
    if X.dtype == np.uint16:                          # bf16 bit patterns
        X = (X.astype(np.uint32) << np.uint32(16)).view(np.float32)
    y = np.asarray(y, dtype=np.int64)
    _, logits = forward(params, X, prec)
    z = logits.astype(np.float64)
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(z - zmax).sum(axis=1))
    row_loss = lse - z[np.arange(z.shape[0]), y]
    pred = np.argmax(logits, axis=1).astype(np.int64)   # first maximum on ties
    return row_loss, pred, logits


# ---------------------------------------------------------------------------
# Flat packing (W_0, b_0, W_1, b_1, ...), the layout of the central variable
# ---------------------------------------------------------------------------

def flat_params(params) -> np.ndarray:
    return np.concatenate([np.concatenate([W.ravel(), b.ravel()]) for W, b in params])


def unflat_params(vec: np.ndarray, dims: Sequence[int], dtype=np.float32):
    out, o = [], 0
    for l in range(len(dims) - 1):
        fi, fo = dims[l], dims[l + 1]
        W = np.array(vec[o:o + fi * fo], dtype=dtype).reshape(fo, fi)
        o += fi * fo
        b = np.array(vec[o:o + fo], dtype=dtype)
        o += fo
        out.append((W, b))
    return out


# ---------------------------------------------------------------------------
# The AGN round: Algorithm 1 for every worker, then Eq. (2) in commit order
# ---------------------------------------------------------------------------

class AGNOracle:
    """n AGN workers and one parameter server, simulated on the CPU.

    State: the central variable, each worker's current parameters, the
    round counter r and, for the staleness check, the server's version
    counter (number of commits applied) and the version each worker last
    pulled.
    """

    def __init__(self, dims, n, lam, eta, m, seed=0, bf16=False, dtype=np.float32,
                 init=None, normalize=True, adam=None, staleness_scaled=False):
        if n < 1 or lam < 1 or m < 1 or len(dims) < 2:
            raise ValueError("bad shapes")
        self.dims = tuple(int(d) for d in dims)
        self.n, self.lam, self.m = int(n), int(lam), int(m)
        # normalize=False: the worker commits its accumulated update itself
        # (Section 2: DOWNPOUR with local exploration, the variant whose
        # divergence motivates the normalization); with lam = 1 both rules
        # are DOWNPOUR (Section 3, footnote to Eq. 1)
        self.normalize = bool(normalize)
        # adam=(beta1, beta2, eps): the local step of Algorithm 1 comes from
        # Adam (Algorithm 1's gradient line names it as an option; Kingma &
        # Ba 2015): per worker first and second moment estimates of its
        # gradients, zero at the start and kept across pulls (the worker's
        # step counter t of Algorithm 1 is not reset by a pull either), and
        # g = -eta * mhat / (sqrt(vhat) + eps) with mhat = m / (1 - beta1^t),
        # vhat = v / (1 - beta2^t) at the worker's local step t = 1, 2, ...
        self.adam = None if adam is None else tuple(float(a) for a in adam)
        # staleness_scaled: the server multiplies each commit by
        # 1 / (tau + 1) (rounded to float32), tau = commits applied since
        # the committing worker's last pull (Section 4's DynSGD rule,
        # scaling commits down by their staleness)
        self.staleness_scaled = bool(staleness_scaled)
        self.prec = _Prec(dtype, bf16)
        self.eta = self.prec.dtype.type(eta)
        if init is None:
            central = he_normal_init(self.dims, seed, dtype=self.prec.dtype)
        else:
            central = [(np.array(W, dtype=self.prec.dtype), np.array(b, dtype=self.prec.dtype))
                       for W, b in init]
        self.central = central
        # Algorithm 1, first line: every worker starts from the pulled central variable
        self.workers = [[(W.copy(), b.copy()) for W, b in central] for _ in range(self.n)]
        if self.adam is not None:
            self.moments = [[(np.zeros_like(W), np.zeros_like(b), np.zeros_like(W), np.zeros_like(b))
                             for W, b in central] for _ in range(self.n)]
        self.r = 0
        self.version = 0
        self.pulled_version = [0] * self.n
        self.staleness: List[List[int]] = []   # per round, in commit order
        self.last_loss = None
        self.last_deltas = None
        # diagnostic for the parity tests (no effect on the arithmetic): when
        # set, round() records per worker the hidden units near a ReLU flip
        # (near_zero_units) over the worker's local steps in last_near
        self.record_near = False
        self.last_near = None

    # -- one worker's lambda local steps (Algorithm 1, inner loop + normalization)
    def _worker_round(self, k, X, y, S):
        st = self.prec.st
        theta = [(W.copy(), b.copy()) for W, b in self.workers[k]]
        a = [(np.zeros_like(W), np.zeros_like(b)) for W, b in theta]
        losses = []
        self._near = [set() for _ in range(len(theta) - 1)]
        for i in range(self.lam):
            t = self.r * self.lam + i
            idx = batch_indices(k, t, self.m, S)           # FetchNextMiniBatch
            if self.record_near:
                for acc, units in zip(self._near, near_zero_units(theta, X[idx], self.prec)):
                    acc.update(int(u) for u in units)
            loss, grads = loss_and_grads(theta, X[idx], y[idx], self.prec)
            losses.append(loss)
            new_theta, new_a = [], []
            for li, ((W, b), (aW, ab), (gW, gb)) in enumerate(zip(theta, a, grads)):
                if self.adam is None:
                    g_W = st(-np.float64(self.eta) * gW)       # g = -eta * grad
                    g_b = st(-np.float64(self.eta) * gb)
                else:
                    g_W, g_b = self._adam_step(k, li, gW, gb, t + 1)
                new_a.append((st(aW + g_W), st(ab + g_b)))           # a <- a + g
                new_theta.append((st(W + g_W), st(b + g_b)))         # theta <- theta + g
            theta, a = new_theta, new_a
        if self.normalize:                                  # the normalization step
            a = [(st(aW / np.float64(self.lam)), st(ab / np.float64(self.lam))) for aW, ab in a]
        return a, float(np.mean(losses)), theta

    def _adam_step(self, k, li, gW, gb, t):
        """Adam's step for worker k, layer li, at the worker's local step t
        (1-based): moments stored in float32, the step in float64, rounded
        once."""
        st = self.prec.st
        b1, b2, eps = (np.float64(x) for x in self.adam)
        mW, mb, vW, vb = self.moments[k][li]
        out = []
        new = []
        for g, mo, ve in ((gW, mW, vW), (gb, mb, vb)):
            g = np.asarray(g, dtype=np.float64)
            m1 = st(b1 * mo + (1.0 - b1) * g)
            v1 = st(b2 * ve + (1.0 - b2) * g * g)
            mhat = m1.astype(np.float64) / (1.0 - b1 ** t)
            vhat = v1.astype(np.float64) / (1.0 - b2 ** t)
            out.append(st(-np.float64(self.eta) * mhat / (np.sqrt(vhat) + eps)))
            new.append((m1, v1))
        self.moments[k][li] = (new[0][0], new[1][0], new[0][1], new[1][1])
        return out[0], out[1]

    def round(self, X, y, order):
        """One AGN round on data (X [N][d_0], y [N]) with the given commit
        order (a permutation of 0..n-1)."""
        order = [int(k) for k in order]
        if sorted(order) != list(range(self.n)):
            raise ValueError("commit order must be a permutation of 0..n-1")
        X = np.asarray(X)
        if X.dtype == np.uint16:                      # bf16 bit patterns
            X = (X.astype(np.uint32) << np.uint32(16)).view(np.float32)
        y = np.asarray(y)
        S = X.shape[0] // self.n
        deltas, losses, finals, near = [], [], [], []
        for k in range(self.n):
            a, loss, theta_fin = self._worker_round(k, X, y, S)
            deltas.append(a)
            losses.append(loss)
            finals.append(theta_fin)
            near.append([np.array(sorted(u), dtype=np.int64) for u in self._near])
        st = self.prec.st
        stale = []
        for k in order:
            tau = self.version - self.pulled_version[k]
            if self.staleness_scaled:
                # central <- central + s * delta_k, s = fl32(1 / (tau + 1)),
                # the product and the sum rounded once
                sc = np.float64(np.float32(1.0 / (tau + 1)))
                self.central = [(st(W + sc * np.asarray(dW, dtype=np.float64)),
                                 st(b + sc * np.asarray(db, dtype=np.float64)))
                                for (W, b), (dW, db) in zip(self.central, deltas[k])]
            else:
                # Commit (Eq. 2): central <- central + delta_k
                self.central = [(st(W + dW), st(b + db))
                                for (W, b), (dW, db) in zip(self.central, deltas[k])]
            stale.append(tau)
            self.version += 1
            # Pull right after the worker's own commit
            self.workers[k] = [(W.copy(), b.copy()) for W, b in self.central]
            self.pulled_version[k] = self.version
        self.staleness.append(stale)
        self.last_loss = np.array(losses, dtype=np.float32)
        self.last_deltas = deltas
        self.last_finals = finals
        self.last_near = near if self.record_near else None
        self.r += 1

    # -- views
    def central_flat(self) -> np.ndarray:
        return flat_params(self.central)

    def worker_flat(self, k) -> np.ndarray:
        return flat_params(self.workers[k])
