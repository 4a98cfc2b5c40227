"""Arithmetic coding of Alg. 1: TEST INFRASTRUCTURE ONLY.

A plain, slow CPU implementation of the coding half of the compressor
(Alg. 1: the first c bytes coded with probability 1/256, every later byte with
the model's estimate; Sec. 3.2 names arithmetic coding after Witten, Neal and
Cleary).  Only the test suite may import it.  It shares no code with the HIP
library and never imports it.

The paper is silent on how the estimate becomes integer code intervals and on
the coder's word size.  Readings used here (and by the library):

* quantisation: for logits z[256] (float32) of one window,
      m = max z,  d_s = (m - z_s) * log2(e)           (float32, IEEE, in this order)
      u_s = trunc(d_s * 256 + 0.5)   if d_s < 32, else 32*256 - 1
      w_s = T[u_s mod 256] >> (u_s div 256),  T[j] = round(2^31 * 2^(-j/256))
      freq_s = 1 + (w_s * 65280) div (sum_r w_r)       (exact integers)
  so w_s is 2^31 * 2^(-d_s) rounded to steps of 2^(1/256) (relative error
  below 0.14 %), every byte keeps a nonzero frequency, and the total is at
  most 65536.  Everything after d_s is exact integer arithmetic, and d_s is
  two correctly rounded float32 operations, so any two implementations that
  follow these steps agree bit for bit;
* the coder: a 32-bit range coder (the arithmetic coder with integer
  renormalisation by bytes): range r, low l (carry into a cached byte),
  encode(cum, f, total): q = r div total, l += q*cum, r = q*f, and while
  r < 2^24 one byte leaves (r <<= 8).  The first byte written is always 0; the
  decoder reads 5 bytes to start and zeros past the end;
* the controller's cross-entropy for a step is the batch mean of the coded
  length log2(total) - log2(freq[x]) in double (both coder sides see it);
* each stream is coded independently (one code per stream of a batch).
"""
from __future__ import annotations

import math
from decimal import Decimal, getcontext

import numpy as np

QBITS_TOTAL = 65536
QSPREAD = 65280          # 65536 - 256: the part of the total spread by weight
QSTEPS = 256             # steps of d per bit
QMAX = 32 * QSTEPS - 1   # largest u (weights below 2^-32 of the top one)
LOG2E_F32 = np.float32(1.4426950408889634)


def quant_table() -> list[int]:
    """T[j] = round(2^31 * 2^(-j/256)), j < 256, from 40-digit decimal
    arithmetic (the values are irrational for j > 0: no ties)."""
    getcontext().prec = 40
    ln2 = Decimal(2).ln()
    out = []
    for j in range(256):
        v = (Decimal(2) ** 31) * (-(Decimal(j) / 256) * ln2).exp()
        out.append(int(v.to_integral_value()))
    return out


_T = None


def quantize(z: np.ndarray) -> np.ndarray:
    """Integer frequencies [..., 256] (int64) of logits z [..., 256] by the
    steps in the module header (the float32 part in float32)."""
    global _T
    if _T is None:
        _T = np.array(quant_table(), dtype=np.uint64)
    z = np.asarray(z, np.float32)
    m = z.max(axis=-1, keepdims=True)
    d = (m - z).astype(np.float32) * LOG2E_F32          # float32 ops
    t = (d * np.float32(256.0)).astype(np.float32) + np.float32(0.5)
    big = ~(d < np.float32(32.0))
    u = np.where(big, QMAX, np.trunc(np.where(big, 0, t))).astype(np.int64)
    u = np.minimum(u, QMAX)
    w = _T[u & 255] >> (u >> 8).astype(np.uint64)
    S = w.sum(axis=-1, keepdims=True, dtype=np.uint64)
    # w * 65280 < 2^47 and S < 2^40: exact in uint64
    return (1 + (w * np.uint64(QSPREAD)) // S).astype(np.int64)


class RangeEncoder:
    """32-bit range coder, encoder side (module header)."""

    def __init__(self):
        self.low = 0
        self.range = 0xFFFFFFFF
        self.cache = 0
        self.pending = 1
        self.out = bytearray()

    def _shift_low(self):
        if self.low < 0xFF000000 or self.low >= (1 << 32):
            carry = self.low >> 32
            byte = self.cache
            while True:
                self.out.append((byte + carry) & 0xFF)
                byte = 0xFF
                self.pending -= 1
                if self.pending == 0:
                    break
            self.cache = (self.low >> 24) & 0xFF
        self.pending += 1
        self.low = (self.low & 0x00FFFFFF) << 8

    def encode(self, cum: int, freq: int, total: int):
        assert 0 < freq and cum + freq <= total <= QBITS_TOTAL
        q = self.range // total
        self.low += q * cum
        self.range = q * freq
        while self.range < (1 << 24):
            self.range <<= 8
            self._shift_low()

    def finish(self) -> bytes:
        for _ in range(5):
            self._shift_low()
        return bytes(self.out)


class RangeDecoder:
    """32-bit range coder, decoder side."""

    def __init__(self, data: bytes):
        self.data = data
        self.pos = 0
        self.range = 0xFFFFFFFF
        self.code = 0
        for _ in range(5):
            self.code = ((self.code << 8) | self._byte()) & 0xFFFFFFFF

    def _byte(self) -> int:
        b = self.data[self.pos] if self.pos < len(self.data) else 0
        self.pos += 1
        return b

    def decode(self, freq) -> int:
        """The symbol whose interval holds the code, for frequencies freq[256]
        (or a shorter alphabet)."""
        total = int(sum(int(f) for f in freq))
        q = self.range // total
        v = min(self.code // q, total - 1)
        cum = 0
        for s, f in enumerate(freq):
            f = int(f)
            if v < cum + f:
                break
            cum += f
        self.code -= q * cum
        self.range = q * f
        while self.range < (1 << 24):
            self.code = ((self.code << 8) | self._byte()) & 0xFFFFFFFF
            self.range <<= 8
        return s


def encode_symbols(freqs, symbols) -> bytes:
    """One code for symbols[i] under frequency row freqs[i]."""
    enc = RangeEncoder()
    for f, x in zip(freqs, symbols):
        f = [int(v) for v in f]
        enc.encode(sum(f[:int(x)]), f[int(x)], sum(f))
    return enc.finish()


def decode_symbols(freqs, data: bytes) -> list[int]:
    dec = RangeDecoder(data)
    return [dec.decode(f) for f in freqs]


UNIFORM = [1] * 256


def coded_bits(freq_row, x) -> float:
    """Coded length of x under one frequency row, log2(total) - log2(freq[x])."""
    return math.log2(int(np.sum(freq_row))) - math.log2(int(freq_row[int(x)]))


# --------------------------------------------- the compressor of Alg. 1 ----
MODE_NEVER, MODE_GATED, MODE_ALWAYS = 0, 1, 2


def _decide(mode, ctl, e):
    if mode == MODE_ALWAYS:
        return 1
    if mode == MODE_GATED:
        return ctl.decide(e)
    return 0


def _run(flat0, cfg, B, L, mode, t, delta, prec, step):
    """The loop shared by both directions: bytes [0, c) under 1/256 (Alg. 1
    lines 1-5), then per position i >= c one forward over the B windows ending
    before i (line 8), the coding step (line 9, step(i, F) returns the bytes at
    i), the controller on the coded length (Alg. 2) and, if it says so, the
    backward + Adam of line 10 on that batch."""
    from . import trace_oracle as O
    W = cfg.W
    theta = np.asarray(flat0, np.float32).copy()
    opt = O.Adam(theta.size, cfg)
    ctl = O.Controller(t, delta)
    decisions = []
    cur = np.zeros((B, L), np.uint8)
    for i in range(min(W, L)):
        cur[:, i] = step(i, None)
    for i in range(W, L):
        w, _ = O.windows_at(cur, np.arange(B), np.full(B, i), W)
        out = O.forward(theta, cfg, w, np.zeros(B, np.int64), mode=prec, keep=False)
        F = quantize(np.asarray(out["z"], np.float32))
        cur[:, i] = step(i, F)
        e = 0.0
        for b in range(B):
            e += coded_bits(F[b], cur[b, i])
        e /= B
        d = _decide(mode, ctl, e)
        decisions.append(d)
        if d:
            w, y = O.windows_at(cur, np.arange(B), np.full(B, i), W)
            out = O.forward(theta, cfg, w, y, mode=prec, keep=True)
            out["windows"] = w
            grads = O.backward(out, cfg)
            theta = opt.step(theta, O.flatten(grads, cfg, np.float32))
    return cur, decisions


def compress(flat0, cfg, streams, mode=MODE_NEVER, t=16, delta=0.05, prec="fp64"):
    """Codes B streams [B][L] of equal length; returns (codes, decisions)."""
    streams = np.asarray(streams, np.uint8)
    B, L = streams.shape
    encs = [RangeEncoder() for _ in range(B)]

    def step(i, F):
        for b in range(B):
            x = int(streams[b, i])
            if F is None:
                encs[b].encode(x, 1, 256)
            else:
                f = F[b]
                encs[b].encode(int(f[:x].sum()), int(f[x]), int(f.sum()))
        return streams[:, i]

    _, dec = _run(flat0, cfg, B, L, mode, t, delta, prec, step)
    return [e.finish() for e in encs], dec


def decompress(flat0, cfg, codes, L, mode=MODE_NEVER, t=16, delta=0.05, prec="fp64"):
    """Inverse of compress: the same loop, each byte taken from its code."""
    B = len(codes)
    decs = [RangeDecoder(c) for c in codes]

    def step(i, F):
        return np.array([decs[b].decode(UNIFORM if F is None else F[b]) for b in range(B)], np.uint8)

    cur, dec = _run(flat0, cfg, B, L, mode, t, delta, prec, step)
    return cur, dec
