// SHA-256 compression for gfx950 (CDNA4), one message per lane.
//
// FIPS 180-4: functions Sec. 4.1.2, constants Sec. 4.2.2 and 5.3.3, message
// schedule and compression Sec. 6.2.2.  The round constants and the initial
// hash value are computed at compile time from their definition (fractional
// parts of the cube / square roots of the first primes), not typed in.
//
// Mapping to the gfx950 vector ALU, one 32-bit op each:
//   rotate right      v_alignbit_b32 x, x, n
//   three-way xor     v_bitop3_b32 (truth table 0x96)
//   majority          v_bitop3_b32 (truth table 0xE8)
//   choose            v_bitop3_b32 (truth table 0xCA)
//   three-input add   v_add3_u32
//   byte swap         v_perm_b32
// so a round is 14 ops (4 for each big sigma, 1 choose, 1 majority, 2 adds
// for T1, 1 add for e, 1 add3 for a) and a schedule word 10 ops.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvgov {

// ---------------------------------------------------------------------------
// constants from their definition
// ---------------------------------------------------------------------------

constexpr bool is_prime(uint32_t v) {
  if (v < 2) return false;
  for (uint32_t d = 2; d * d <= v; ++d)
    if (v % d == 0) return false;
  return true;
}

constexpr uint32_t nth_prime(int n) {  // n = 0 -> 2
  uint32_t v = 1;
  for (int c = -1; c < n;) {
    ++v;
    if (is_prime(v)) ++c;
  }
  return v;
}

// floor(v^(1/k)) by bisection; k in {2, 3}, v < 2^110
constexpr unsigned __int128 iroot(unsigned __int128 v, int k) {
  unsigned __int128 lo = 0, hi = (unsigned __int128)1 << 37;
  while (lo < hi) {
    unsigned __int128 mid = (lo + hi + 1) / 2;
    unsigned __int128 p = mid * mid;
    if (k == 3) p *= mid;
    if (p <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// first 32 bits of the fractional part of p^(1/k)
constexpr uint32_t frac32(uint32_t p, int k) {
  return (uint32_t)iroot((unsigned __int128)p << (32 * k), k);
}

struct Sha256Tables {
  uint32_t K[64];
  uint32_t H0[8];
};

constexpr Sha256Tables make_tables() {
  Sha256Tables t{};
  for (int i = 0; i < 64; ++i) t.K[i] = frac32(nth_prime(i), 3);
  for (int i = 0; i < 8; ++i) t.H0[i] = frac32(nth_prime(i), 2);
  return t;
}

inline constexpr Sha256Tables kSha = make_tables();

static_assert(kSha.K[0] == frac32(2, 3) && kSha.H0[7] == frac32(19, 2), "tables");

// ---------------------------------------------------------------------------
// primitives
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t rotr(uint32_t x, uint32_t n) {
  return __builtin_amdgcn_alignbit(x, x, n);
}
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}
__device__ __forceinline__ uint32_t maj(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0xE8);
}
__device__ __forceinline__ uint32_t ch(uint32_t e, uint32_t f, uint32_t g) {
  return __builtin_amdgcn_bitop3_b32(e, f, g, 0xCA);
}
__device__ __forceinline__ uint32_t big_sigma0(uint32_t x) {
  return xor3(rotr(x, 2), rotr(x, 13), rotr(x, 22));
}
__device__ __forceinline__ uint32_t big_sigma1(uint32_t x) {
  return xor3(rotr(x, 6), rotr(x, 11), rotr(x, 25));
}
__device__ __forceinline__ uint32_t small_sigma0(uint32_t x) {
  return xor3(rotr(x, 7), rotr(x, 18), x >> 3);
}
__device__ __forceinline__ uint32_t small_sigma1(uint32_t x) {
  return xor3(rotr(x, 17), rotr(x, 19), x >> 10);
}
// little-endian int32 token <-> big-endian message word
__device__ __forceinline__ uint32_t bswap(uint32_t x) {
  return __builtin_amdgcn_perm(x, x, 0x00010203u);
}

__device__ __forceinline__ void set_iv(uint32_t st[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) st[i] = kSha.H0[i];
}

// One compression: st <- st + rounds(st, w).  w[16] is the message block as
// big-endian words; it is overwritten by the rolling schedule.
__device__ __forceinline__ void compress(uint32_t st[8], uint32_t w[16]) {
  uint32_t a = st[0], b = st[1], c = st[2], d = st[3];
  uint32_t e = st[4], f = st[5], g = st[6], h = st[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    if (t >= 16) {
      w[t & 15] = small_sigma1(w[(t - 2) & 15]) + w[(t - 7) & 15] +
                  small_sigma0(w[(t - 15) & 15]) + w[t & 15];
    }
    const uint32_t t1 = h + big_sigma1(e) + ch(e, f, g) + kSha.K[t] + w[t & 15];
    const uint32_t t2 = big_sigma0(a) + maj(a, b, c);
    h = g;
    g = f;
    f = e;
    e = d + t1;
    d = c;
    c = b;
    b = a;
    a = t1 + t2;
  }
  st[0] += a; st[1] += b; st[2] += c; st[3] += d;
  st[4] += e; st[5] += f; st[6] += g; st[7] += h;
}

}  // namespace kvgov
