"""TRACE oracle: TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct CPU implementation of the TRACE next-byte
estimator and its gated online update (Mao et al., "A Fast Transformer-based
General-Purpose Lossless Compressor", arXiv 2203.16114).  It exists to check
the HIP path; only the test suite, the package's smoke check and the CPU
baseline leg of the benchmark may import it.  It shares no code with the HIP
library and never imports it.

Every function cites the passage it follows.  Where the paper is silent the
reading used is stated next to the code:

* window and grouping (Sec. 4.2; Alg. 1): the estimate for byte x_i reads the
  W = c*g previous bytes, oldest first; byte j of group t fills dims
  [j*e, (j+1)*e) of token t (oldest byte in the lowest dims);
* a learned positional table P[T][d] is added after grouping (paper silent);
* attention (Eqs. 1-2) is causal, per head with scale 1/sqrt(d/H), heads
  concatenated in order and projected by Wo; no biases, no LayerNorm (Eq. 4);
* the layer (Eq. 4) with the shared FFN of Sec. 4.3:
  Y0 = Attn(X) + X,  Y_r = Y_{r-1} + GELU(Y_{r-1} W1) W2 (r = 1..k);
* the 256-way head reads the last token: z = Y_k[T-1] Wout + bout, and the code
  length of the target is -log2 softmax(z)[y];
* the loss for the update is the batch-mean cross-entropy in nats;
* Adam (Kingma & Ba 2015, Alg. 1) with bias correction, step count advanced
  only on applied updates;
* the back-prop controller (Sec. 4.4, Alg. 2, Eq. 7) updates iff the step's
  mean code length exceeds the mean of the last t values plus delta, and
  always during the first t steps.

Precision modes: "fp64" (reference for fp32 work and for the finite-difference
pins), "fp32", and "bf16" = fp32 arithmetic with round-to-nearest-even to
bfloat16 at the storage points listed above ``compute_params``.

Parity pins for every function live in tests/test_oracle_*.py.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
from scipy.special import erfc as _erfc

LOG2E = 1.0 / math.log(2.0)


# ---------------------------------------------------------------- config ----
@dataclass(frozen=True)
class Config:
    """Model shape (Sec. 4, Fig. 2/4): window W bytes, per-byte width e, group g,
    heads H, FFN width F, shared-FFN repeats k."""

    W: int
    e: int
    g: int
    H: int
    F: int
    k: int
    use_pos: bool = True
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    # False: the k repeats share W1, W2 (Sec. 4.3); True: one W1, W2 per repeat
    # (the deep-FFN variant of Sec. 6.3), stored as k consecutive blocks
    untied: bool = False
    # "softmax": Eqs. 1-2; "performer": the FAVOR+ attention of the Performer
    # the paper's experiments use as backbone (Sec. 6), with n_features random
    # features (the projection matrix is an input of forward)
    attention: str = "softmax"
    n_features: int = 0
    # layers of Eq. 4 stacked (Sec. 6.3, Fig. 7); every layer has its own
    # Wq, Wk, Wv, Wo, W1, W2, stored as `layers` consecutive blocks of each
    layers: int = 1

    @property
    def T(self) -> int:  # tokens per window (Sec. 4.2: c groups)
        return self.W // self.g

    @property
    def d(self) -> int:  # token width h = g * (h/g)
        return self.g * self.e

    @property
    def dh(self) -> int:  # per-head width
        return self.d // self.H

    @property
    def m(self) -> int:  # Performer random features (reading: about dh ln dh, a multiple of 64)
        return self.n_features or (128 if self.dh <= 32 else 256)


def param_layout(cfg: Config):
    """Canonical flat parameter order, each matrix row-major [in][out]."""
    T, d, e, F = cfg.T, cfg.d, cfg.e, cfg.F
    Ls = (cfg.layers,) if cfg.layers > 1 else ()
    return [
        ("E", (256, e)),
        ("P", (T, d)),
        ("Wq", Ls + (d, d)),
        ("Wk", Ls + (d, d)),
        ("Wv", Ls + (d, d)),
        ("Wo", Ls + (d, d)),
        ("W1", Ls + ((cfg.k, d, F) if cfg.untied else (d, F))),
        ("W2", Ls + ((cfg.k, F, d) if cfg.untied else (F, d))),
        ("Wout", (d, 256)),
        ("bout", (256,)),
    ]


_LAYER_WEIGHTS = ("Wq", "Wk", "Wv", "Wo", "W1", "W2")


def layer_params(p: dict, cfg: Config, l: int) -> dict:
    """Layer l's Wq .. W2 (views into p, or p's own arrays when layers = 1)."""
    return {n: (p[n][l] if cfg.layers > 1 else p[n]) for n in _LAYER_WEIGHTS}


def param_count(cfg: Config) -> int:
    return sum(int(np.prod(s)) for _, s in param_layout(cfg))


def unflatten(flat: np.ndarray, cfg: Config) -> dict:
    """Views into the flat buffer, by name."""
    out, off = {}, 0
    for name, shape in param_layout(cfg):
        n = int(np.prod(shape))
        out[name] = flat[off:off + n].reshape(shape)
        off += n
    assert off == flat.size
    return out


def flatten(p: dict, cfg: Config, dtype=np.float64) -> np.ndarray:
    return np.concatenate([np.asarray(p[n], dtype).ravel() for n, _ in param_layout(cfg)])


# ---------------------------------------------------------- initialisation ----
_M64 = (1 << 64) - 1


def splitmix64(state: int):
    """One step of Vigna's splitmix64; returns (new_state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & _M64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return state, z ^ (z >> 31)


def init_flat(cfg: Config, seed: int, std: float = 0.02) -> np.ndarray:
    """Model.initialize() of Alg. 1 (random start, Sec. 5 "Dynamic-Random").

    Every entry of E, P, Wq..Wout is std*N(0,1) drawn by Box-Muller from
    splitmix64 uniforms u = ((x >> 11) + 0.5) * 2^-53, in the flat order;
    bout = 0.  Scalar libm calls (math.log/cos/sin/sqrt) so that a C library
    calling the same libm reproduces the values bit for bit."""
    n_total = param_count(cfg)
    n_rand = n_total - 256  # bout is last and zero
    out = np.zeros(n_total, np.float32)
    state = seed & _M64
    two_pi = 2.0 * math.pi
    i = 0
    while i < n_rand:
        state, x1 = splitmix64(state)
        state, x2 = splitmix64(state)
        u1 = ((x1 >> 11) + 0.5) * (2.0 ** -53)
        u2 = ((x2 >> 11) + 0.5) * (2.0 ** -53)
        r = math.sqrt(-2.0 * math.log(u1))
        out[i] = np.float32(std * (r * math.cos(two_pi * u2)))
        if i + 1 < n_rand:
            out[i + 1] = np.float32(std * (r * math.sin(two_pi * u2)))
        i += 2
    return out


# --------------------------------------------------------------- rounding ----
def bf16_round(x) -> np.ndarray:
    """fp32 -> bfloat16 -> fp32 with round-to-nearest-even (NaN preserved).

    Adds 0x7FFF plus the lowest kept bit, then clears the 16 low bits.  In
    32-bit unsigned arithmetic only NaN patterns (0xFFFF7FFF and above) wrap;
    NaNs are restored from the input afterwards."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)) << np.uint32(16)
    out = r.view(np.float32)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = x[nan]
    return out


class _Mode:
    """Arithmetic type and storage-point rounding for one precision mode."""

    def __init__(self, mode: str):
        if mode not in ("fp64", "fp32", "bf16"):
            raise ValueError(mode)
        self.name = mode
        self.dt = np.float64 if mode == "fp64" else np.float32

    def R(self, x):
        """Storage point: rounds to bf16 in bf16 mode, else a cast."""
        x = np.asarray(x, self.dt)
        return bf16_round(x) if self.name == "bf16" else x

    def A(self, x):
        return np.asarray(x, self.dt)


# bf16 storage points (all else fp32): the weight copies E,P,Wq,Wk,Wv,Wo,W1,W2,
# Wout; the GEMM operands O, Y_{r-1} (into W1), GELU(U_r) (into W2), Y_k (into
# the head); in the backward dz, dY, dU, dO.  The token X = E[byte] + P[t] is
# not one: it is the fp32 sum of two rounded copies, and the projections take it
# as it is (X.W = E.W + P.W exactly, which lets the projection of a byte group be
# shared by every window that holds it).
_WEIGHTS_ROUNDED = ("E", "P", "Wq", "Wk", "Wv", "Wo", "W1", "W2", "Wout")


def compute_params(flat: np.ndarray, cfg: Config, mode: str) -> dict:
    m = _Mode(mode)
    p = unflatten(np.asarray(flat), cfg)
    q = {}
    for name, _ in param_layout(cfg):
        q[name] = m.R(p[name]) if name in _WEIGHTS_ROUNDED else m.A(p[name])
    return q


# ------------------------------------------------------------ primitives ----
def _Phi(u):
    """Standard normal CDF, 0.5 * erfc(-u / sqrt 2) (no cancellation in the tail)."""
    dt = u.dtype
    return 0.5 * _erfc(-u / np.sqrt(dt.type(2.0)))


def gelu(u):
    """Eq. 3's GELU, exact erf form: u * Phi(u) = 0.5 u (1 + erf(u / sqrt 2))."""
    return (u * _Phi(u)).astype(u.dtype)


def gelu_grad(u):
    """d/du [u Phi(u)] = Phi(u) + u phi(u)."""
    dt = u.dtype
    Phi = _Phi(u)
    phi = np.exp(-0.5 * u * u) / np.sqrt(dt.type(2.0 * math.pi))
    return (Phi + u * phi).astype(dt)


def softmax_lastaxis(s):
    m = np.max(s, axis=-1, keepdims=True)
    ex = np.exp(s - m)
    return ex / np.sum(ex, axis=-1, keepdims=True)


# ------------------------------------------------------------------ windows ----
def windows_at(streams: np.ndarray, b: np.ndarray, i: np.ndarray, W: int):
    """Alg. 1 line 8: the context of target x_i is x_{i-W} .. x_{i-1} (oldest
    first); returns (windows [N][W] uint8, targets [N] uint8)."""
    b = np.asarray(b, np.int64)
    i = np.asarray(i, np.int64)
    if np.any(i < W):
        raise ValueError("targets before position W have no full window")
    cols = i[:, None] - W + np.arange(W)[None, :]
    return streams[b[:, None], cols], streams[b, i]


def all_windows(streams: np.ndarray, W: int, pos0: int | None = None, n_steps: int | None = None):
    """Every window of every stream for targets pos0 .. pos0+n_steps-1, ordered
    [stream][step]."""
    B, L = streams.shape
    pos0 = W if pos0 is None else pos0
    n_steps = L - pos0 if n_steps is None else n_steps
    bb, ii = np.meshgrid(np.arange(B), pos0 + np.arange(n_steps), indexing="ij")
    return windows_at(streams, bb.ravel(), ii.ravel(), W)


# ------------------------------------------------------------------ forward ----
def embed_group(p: dict, windows: np.ndarray, cfg: Config, m: _Mode):
    """Sec. 4.2 byte-grouping: each byte becomes an e-vector E[byte]; bytes
    t*g .. t*g+g-1 are concatenated (oldest first) into token t of width d.
    Returns X as fp (residual copy; positional table added when use_pos)."""
    N = windows.shape[0]
    X = np.zeros((N, cfg.T, cfg.d), m.dt)
    for t in range(cfg.T):
        for j in range(cfg.g):
            X[:, t, j * cfg.e:(j + 1) * cfg.e] = p["E"][windows[:, t * cfg.g + j]]
    if cfg.use_pos:
        X = X + p["P"][None, :, :]
    return X


def performer_attention_weights(Qh, Kh, omega, dt):
    """Causal FAVOR+ attention weights (Performer, Choromanski et al. 2021) for
    one head: the softmax kernel exp(q.k / sqrt(dh)) of Eq. 1 is replaced by
    phi(q')^T phi(k') with positive random features phi(x) = m^-1/2 exp(omega x
    - |x|^2/2) of the scaled q' = q dh^-1/4, k' = k dh^-1/4 (so q'.k' =
    q.k/sqrt(dh)), omega [m][dh].  Row t of A is phi(q'_t)^T phi(k'_u)
    normalised over u <= t.  phi is taken relative to a constant per query
    row (max over features) and per window for the keys (max over keys and
    features), constants that cancel in the normalisation.
    Qh, Kh [N][T][dh] -> A [N][T][T]."""
    N, T, dh = Qh.shape
    s4 = dt(dh ** -0.25)
    qs, ks = Qh * s4, Kh * s4
    pq = qs @ omega.T - dt(0.5) * np.sum(qs * qs, axis=-1, keepdims=True)      # [N][T][m]
    pk = ks @ omega.T - dt(0.5) * np.sum(ks * ks, axis=-1, keepdims=True)
    fq = np.exp(pq - np.max(pq, axis=-1, keepdims=True))
    fk = np.exp(pk - np.max(pk, axis=(1, 2), keepdims=True))
    kern = np.einsum("ntm,num->ntu", fq, fk)
    kern = np.where(np.tril(np.ones((T, T), bool))[None], kern, dt(0))
    return (kern / np.sum(kern, axis=-1, keepdims=True)).astype(dt)


def layer_forward(q: dict, X, Xo, cfg: Config, m, om=None) -> dict:
    """One layer of Eq. 4 over all T rows (causal): attention of Eqs. 1-2 (or
    the Performer's) on the GEMM operand Xo with the residual X, then the FFN
    of Eq. 3 k times (Sec. 4.3; untied per repeat for Sec. 6.3).  q holds the
    layer's (rounded) weights.  Returns every intermediate; Y[-1] is the
    layer's output."""
    N, T, d, H, dh = X.shape[0], cfg.T, cfg.d, cfg.H, cfg.dh
    Q = Xo @ q["Wq"]
    K = Xo @ q["Wk"]
    V = Xo @ q["Wv"]
    scale = m.dt(1.0 / math.sqrt(dh))                   # Eq. 1, per head
    causal = np.tril(np.ones((T, T), bool))
    A = np.zeros((N, H, T, T), m.dt)
    O = np.zeros((N, T, d), m.dt)
    for h in range(H):
        c = slice(h * dh, (h + 1) * dh)
        if cfg.attention == "performer":
            Ah = performer_attention_weights(Q[:, :, c], K[:, :, c], om, m.dt)
        else:
            S = np.einsum("ntc,nuc->ntu", Q[:, :, c], K[:, :, c]) * scale
            S = np.where(causal[None], S, -np.inf)
            Ah = softmax_lastaxis(S).astype(m.dt)
        A[:, h] = Ah
        O[:, :, c] = np.einsum("ntu,nuc->ntc", Ah, V[:, :, c])
    Oo = m.R(O)
    Attn = Oo @ q["Wo"]                                 # Eq. 2 projection W
    Y = [Attn + X]                                      # Eq. 4 inner residual
    U, Yop, Gop = [], [], []
    for r in range(cfg.k):                              # Sec. 4.3, shared W1, W2 (Sec. 6.3: untied)
        W1r = q["W1"][r] if cfg.untied else q["W1"]
        W2r = q["W2"][r] if cfg.untied else q["W2"]
        yo = m.R(Y[-1])
        u = yo @ W1r
        go = m.R(gelu(u))
        Y.append(Y[-1] + go @ W2r)
        U.append(u); Yop.append(yo); Gop.append(go)
    return dict(X=X, Xo=Xo, Q=Q, K=K, V=V, A=A, O=O, Oo=Oo, Y=Y, U=U, Yop=Yop, Gop=Gop)


def forward(flat: np.ndarray, cfg: Config, windows: np.ndarray, targets: np.ndarray,
            mode: str = "fp64", keep: bool = False, features=None):
    """Model.forward of Alg. 1 line 8: byte grouping (Sec. 4.2), then
    cfg.layers layers of Eqs. 1-4 with the shared FFN of Sec. 4.3, each over
    ALL T rows with a causal mask, and the head on the last row.  Layer 0's
    projections take the token X = E + P as it is; later layers take their
    input (the residual stream) rounded like the FFN's input (a bf16 storage
    point).  Returns dict with logits z [N][256], bits [N] (= -log2
    p(target)), and, if keep, every intermediate (per layer in "layers"; with
    one layer also at the top level).  With cfg.attention == "performer",
    `features` is the random projection omega [m][dh] (one for all heads and
    layers; rounded like a weight copy in bf16 mode)."""
    m = _Mode(mode)
    p = compute_params(flat, cfg, mode)
    windows = np.asarray(windows, np.uint8)
    targets = np.asarray(targets, np.int64)
    T, dh = cfg.T, cfg.dh
    om = None
    if cfg.attention == "performer":
        if features is None or np.shape(features) != (cfg.m, dh):
            raise ValueError("performer attention needs features of shape [m][dh]")
        om = m.R(np.asarray(features, np.float32))
    elif cfg.attention != "softmax":
        raise ValueError(cfg.attention)
    X = embed_group(p, windows, cfg, m)                 # residual copy
    layers = []
    for l in range(cfg.layers):
        Xo = X if l == 0 else m.R(X)                    # layer 0: fp32 token, not rounded
        c = layer_forward(layer_params(p, cfg, l), X, Xo, cfg, m, om)
        layers.append(c)
        X = c["Y"][-1]
    hk = m.R(X[:, T - 1, :])
    z = hk @ p["Wout"] + p["bout"]
    bits = code_length_bits(z, targets)
    out = {"z": z, "bits": bits}
    if keep:
        out.update(dict(p=p, layers=layers, hk=hk, targets=targets, mode=mode))
        if cfg.layers == 1:
            out.update(layers[0])
    return out


def code_length_bits(z: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Alg. 2 line 3 with a one-hot ground truth: e = H(gt) + KL(gt||P) =
    -log2 P(y), with P = softmax(z).  Evaluated stably as
    log2(sum exp(z - max z)) - (z_y - max z) * log2(e)."""
    dt = z.dtype
    mx = np.max(z, axis=1)
    lse = np.log2(np.sum(np.exp(z - mx[:, None]), axis=1))
    zy = z[np.arange(z.shape[0]), y]
    return (lse - (zy - mx) * dt.type(LOG2E)).astype(dt)


def bits_per_byte(bits: np.ndarray) -> float:
    """Model bits/byte: mean code length over every predicted byte."""
    return float(np.mean(np.asarray(bits, np.float64)))


def stream_bits_per_byte(bits_sum: float, B: int, L: int, W: int) -> float:
    """Whole-stream bits/byte charging the first W bytes of each stream 8 bits
    each (Alg. 1 lines 2-5 code them at probability 1/256)."""
    return (8.0 * W * B + bits_sum) / (B * L)


# ----------------------------------------------------------------- backward ----
def layer_backward(c: dict, q: dict, dY, cfg: Config, m) -> tuple:
    """Gradients of one layer (the forward of layer_forward) given dY, the
    gradient w.r.t. its output Y_k (all rows): returns (the layer's weight
    gradients, the gradient w.r.t. its input X)."""
    N, T, d, H, dh = c["X"].shape[0], cfg.T, cfg.d, cfg.H, cfg.dh
    g = {"W1": np.zeros_like(q["W1"]), "W2": np.zeros_like(q["W2"])}
    # shared FFN, repeats in reverse; W1, W2 gradients accumulate over repeats
    for r in reversed(range(cfg.k)):
        # untied: repeat r's own blocks (views, so += lands in g)
        gW1, gW2 = (g["W1"][r], g["W2"][r]) if cfg.untied else (g["W1"], g["W2"])
        W1r, W2r = (q["W1"][r], q["W2"][r]) if cfg.untied else (q["W1"], q["W2"])
        dYo = m.R(dY)
        gW2 += np.einsum("ntf,ntc->fc", c["Gop"][r], dYo)
        dG = dYo @ W2r.T
        dU = dG * gelu_grad(c["U"][r])
        dUo = m.R(dU)
        gW1 += np.einsum("ntc,ntf->cf", c["Yop"][r], dUo)
        dY = dY + dUo @ W1r.T
    dY0 = dY
    dY0o = m.R(dY0)
    g["Wo"] = np.einsum("ntc,nto->co", c["Oo"], dY0o)
    dO = m.R(dY0o @ q["Wo"].T)
    # attention (Eq. 1 per head)
    scale = m.dt(1.0 / math.sqrt(dh))
    dQ = np.zeros((N, T, d), m.dt)
    dK = np.zeros((N, T, d), m.dt)
    dV = np.zeros((N, T, d), m.dt)
    for h in range(H):
        cs = slice(h * dh, (h + 1) * dh)
        Ah = c["A"][:, h]
        dA = np.einsum("ntc,nuc->ntu", dO[:, :, cs], c["V"][:, :, cs])
        dV[:, :, cs] = np.einsum("ntu,ntc->nuc", Ah, dO[:, :, cs])
        dS = Ah * (dA - np.sum(dA * Ah, axis=-1, keepdims=True))
        dQ[:, :, cs] = np.einsum("ntu,nuc->ntc", dS, c["K"][:, :, cs]) * scale
        dK[:, :, cs] = np.einsum("ntu,ntc->nuc", dS, c["Q"][:, :, cs]) * scale
    Xo = c["Xo"]
    g["Wq"] = np.einsum("ntc,nto->co", Xo, dQ)
    g["Wk"] = np.einsum("ntc,nto->co", Xo, dK)
    g["Wv"] = np.einsum("ntc,nto->co", Xo, dV)
    dX = dQ @ q["Wq"].T + dK @ q["Wk"].T + dV @ q["Wv"].T + dY0
    return g, dX


def backward(cache: dict, cfg: Config) -> dict:
    """Gradient of L = (1/N) sum_n CE_nats[n] w.r.t. every parameter (Alg. 1
    line 10), by the chain rule through the forward above, layer by layer from
    the top.  All T rows are carried; only the last row of the top layer's
    output receives an upstream gradient from the head."""
    if cfg.attention != "softmax":
        raise NotImplementedError("the backward covers softmax attention (Eqs. 1-2) only")
    m = _Mode(cache["mode"])
    p = cache["p"]
    layers = cache["layers"]
    N, T, d = layers[0]["X"].shape[0], cfg.T, cfg.d
    y = cache["targets"]
    z = cache["z"]
    g = {}
    # head: softmax cross-entropy in nats
    Pz = softmax_lastaxis(z).astype(m.dt)
    onehot = np.zeros_like(Pz)
    onehot[np.arange(N), y] = 1
    dz = (Pz - onehot) / m.dt(N)
    dzo = m.R(dz)
    g["Wout"] = cache["hk"].T @ dzo
    g["bout"] = dz.sum(axis=0)
    dX = np.zeros((N, T, d), m.dt)
    dX[:, T - 1, :] = dzo @ p["Wout"].T
    for n in _LAYER_WEIGHTS:
        g[n] = np.zeros_like(p[n])
    for l in reversed(range(cfg.layers)):
        gl, dX = layer_backward(layers[l], layer_params(p, cfg, l), dX, cfg, m)
        dst = layer_params(g, cfg, l)
        for n in _LAYER_WEIGHTS:
            dst[n][...] = gl[n]
    g["P"] = dX.sum(axis=0) if cfg.use_pos else np.zeros_like(p["P"])
    # embedding: byte j of token t read E[w] into dims [j*e, (j+1)*e)
    gE = np.zeros_like(p["E"])
    w = cache["windows"] if "windows" in cache else None
    if w is None:
        raise KeyError("cache needs the windows (use forward_backward)")
    for t in range(T):
        for j in range(cfg.g):
            np.add.at(gE, w[:, t * cfg.g + j], dX[:, t, j * cfg.e:(j + 1) * cfg.e])
    g["E"] = gE
    return g


def forward_backward(flat, cfg, windows, targets, mode="fp64"):
    """Forward with activations kept, then the gradient; returns (out, grads)."""
    out = forward(flat, cfg, windows, targets, mode=mode, keep=True)
    out["windows"] = np.asarray(windows, np.uint8)
    return out, backward(out, cfg)


def loss_nats(flat, cfg, windows, targets, mode="fp64") -> float:
    """L = mean cross-entropy in nats over the batch (= ln2 * mean bits)."""
    b = forward(flat, cfg, windows, targets, mode=mode)["bits"]
    return float(np.mean(np.asarray(b, np.float64)) * math.log(2.0))


# --------------------------------------------------------------------- Adam ----
class Adam:
    """Adam (Kingma & Ba 2015, Alg. 1) on the flat fp32 master buffer, lr from
    Sec. 6 (0.001).  tau counts applied updates only."""

    def __init__(self, n: int, cfg: Config):
        self.m = np.zeros(n, np.float32)
        self.v = np.zeros(n, np.float32)
        self.tau = 0
        self.cfg = cfg

    def step(self, theta: np.ndarray, grad: np.ndarray) -> np.ndarray:
        c = self.cfg
        g = np.asarray(grad, np.float32)
        self.tau += 1
        b1, b2 = np.float32(c.beta1), np.float32(c.beta2)
        self.m = b1 * self.m + (np.float32(1) - b1) * g
        self.v = b2 * self.v + (np.float32(1) - b2) * g * g
        bc1 = np.float32(1.0 - c.beta1 ** self.tau)
        bc2 = np.float32(1.0 - c.beta2 ** self.tau)
        mhat = self.m / bc1
        vhat = self.v / bc2
        return (theta - np.float32(c.lr) * mhat / (np.sqrt(vhat) + np.float32(c.eps))).astype(np.float32)


# --------------------------------------------------------------- controller ----
class Controller:
    """Back-prop controller of Sec. 4.4 / Alg. 2 with uniform weights (Eq. 7).

    A FIFO of the last t step cross-entropies (bits) and their running sum.
    decide(e) returns 1 (back-propagate) iff e > S/t + delta, in IEEE double
    with a strict comparison; during the first t steps it returns 1.  The cache
    takes e whatever the decision."""

    def __init__(self, t: int, delta: float):
        if not (1 <= t <= 256):
            raise ValueError("t must be in 1..256")
        self.t, self.delta = t, float(delta)
        self.ring = []
        self.S = 0.0

    def threshold(self) -> float:
        return self.S / self.t + self.delta

    def decide(self, e: float) -> int:
        e = float(e)
        if not math.isfinite(e):
            raise ValueError("non-finite cross-entropy")
        if len(self.ring) < self.t:
            upd = 1
        else:
            upd = 1 if e > (self.S / self.t + self.delta) else 0
        if len(self.ring) == self.t:
            self.S = self.S - self.ring.pop(0)
        self.S = self.S + e
        self.ring.append(e)
        return upd


# ----------------------------------------------------- gated adaptation loop ----
def run_gated(flat0, cfg, streams, pos0, n_steps, t, delta, mode="fp64",
              forced_decisions=None, logits_out=None):
    """Alg. 1 with the controller of Alg. 2 over a batch of B streams: at each
    step every stream predicts its next byte (one window per stream), the
    batch-mean code length e goes to the controller, and if it says so one
    backward + Adam step runs on that same batch.  forced_decisions replays a
    given decision sequence (teacher forcing) instead of the controller's.
    Returns (bits [B][n_steps], step_ce [n_steps], decisions, own decisions,
    final flat fp32 master); if logits_out is a list, each step's logits
    [B][256] are appended to it."""
    B = streams.shape[0]
    theta = np.asarray(flat0, np.float32).copy()
    opt = Adam(theta.size, cfg)
    ctl = Controller(t, delta)
    bits = np.zeros((B, n_steps), np.float64)
    step_ce = np.zeros(n_steps, np.float64)
    dec, own = [], []
    for s in range(n_steps):
        i = pos0 + s
        w, y = windows_at(streams, np.arange(B), np.full(B, i), cfg.W)
        out = forward(theta, cfg, w, y, mode=mode, keep=True)
        out["windows"] = w
        bits[:, s] = out["bits"]
        if logits_out is not None:
            logits_out.append(np.array(out["z"], copy=True))
        e = float(np.mean(np.asarray(out["bits"], np.float64)))
        step_ce[s] = e
        o = ctl.decide(e)
        own.append(o)
        d = o if forced_decisions is None else int(forced_decisions[s])
        dec.append(d)
        if d:
            grads = backward(out, cfg)
            theta = opt.step(theta, flatten(grads, cfg, np.float32))
    return bits, step_ce, dec, own, theta
