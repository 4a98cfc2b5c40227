// Coding of Alg. 1 (lines 3 and 9): integer code intervals from the estimate
// and a 32-bit range coder (an arithmetic coder with integer renormalisation
// by bytes; the paper names arithmetic coding after Witten, Neal and Cleary).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

// frequencies of one window: 256 values >= 1 whose total is at most 65536
constexpr uint32_t QSPREAD = 65280;       // 65536 - 256: the part spread by weight
constexpr int QMAX = 32 * 256 - 1;        // largest fixed-point distance from the top logit

// T[j] = round(2^31 * 2^(-j/256)), j < 256 (host, computed once)
const uint32_t* quant_table();
// freq[w][s] for logits z[w][256] of n windows (device), on stream s
void launch_quantize(const float* z, int64_t n, uint16_t* freq, hipStream_t s);
// dst[b*stride + col] = src[b], b < n (device)
void launch_put_column(const uint8_t* src, int64_t n, uint8_t* dst, int64_t stride, int64_t col, hipStream_t s);

// Encoder: low carries into the byte held back in cache (and the run of 0xFF
// bytes behind it); the first byte written is 0.  Bytes past cap are counted
// but not stored (over).
struct RcEnc {
  uint64_t low = 0;
  uint32_t range = 0xFFFFFFFFu;
  uint8_t cache = 0;
  uint64_t pending = 1;
  uint8_t* out = nullptr;
  int64_t cap = 0, n = 0;

  void put(uint8_t b) {
    if (n < cap) out[n] = b;
    ++n;
  }
  void shift_low() {
    if ((uint32_t)low < 0xFF000000u || (low >> 32) != 0) {
      const uint8_t carry = (uint8_t)(low >> 32);
      uint8_t b = cache;
      do {
        put((uint8_t)(b + carry));
        b = 0xFF;
      } while (--pending != 0);
      cache = (uint8_t)(low >> 24);
    }
    ++pending;
    low = (low & 0x00FFFFFFu) << 8;
  }
  // the symbol with cumulative frequency cum, frequency f, of total <= 2^16
  void encode(uint32_t cum, uint32_t f, uint32_t total) {
    const uint32_t q = range / total;
    low += (uint64_t)q * cum;
    range = q * f;
    while (range < (1u << 24)) {
      range <<= 8;
      shift_low();
    }
  }
  void finish() {
    for (int i = 0; i < 5; ++i) shift_low();
  }
  bool over() const { return n > cap; }
};

// Decoder: reads 5 bytes to start, zeros past the end of the code.
struct RcDec {
  const uint8_t* in = nullptr;
  int64_t size = 0, pos = 0;
  uint32_t range = 0xFFFFFFFFu, code = 0;

  uint32_t next() { return pos < size ? in[pos++] : (++pos, 0u); }
  void start() {
    for (int i = 0; i < 5; ++i) code = (code << 8) | next();
  }
  // the symbol whose interval holds the code, among nsym frequencies f of total
  int decode(const uint16_t* f, int nsym, uint32_t total) {
    const uint32_t q = range / total;
    uint32_t v = code / q;
    if (v >= total) v = total - 1;
    uint32_t cum = 0;
    int s = 0;
    for (; s < nsym - 1; ++s) {
      if (v < cum + f[s]) break;
      cum += f[s];
    }
    code -= q * cum;
    range = q * f[s];
    while (range < (1u << 24)) {
      code = (code << 8) | next();
      range <<= 8;
    }
    return s;
  }
  // a byte of probability 1/256
  int decode_uniform() {
    const uint32_t q = range / 256;
    uint32_t v = code / q;
    if (v > 255) v = 255;
    code -= q * v;
    range = q;
    while (range < (1u << 24)) {
      code = (code << 8) | next();
      range <<= 8;
    }
    return (int)v;
  }
};
