// Salts (HMAC-SHA256) and chained block hashes on gfx950.
//
// Paper: per-principal salt sigma_p = HMAC_K(principal_id) (Sec. 4.1); block
// hashes chained h_j = H(h_{j-1}, tokens_j) (Sec. 2.1) with the salt at the
// root (Sec. 4.1) or at the divergence boundary k (Sec. 4.2).
//
// Execution model.  A chain is a strict sequence of SHA-256 compressions
// (h_j needs h_{j-1}), so one lane owns one request and walks its chain; a
// wave therefore advances 64 chains at once, and all parallelism comes from
// the batch.  Requests are ordered longest first (LPT) so that the 64 lanes
// of a wave carry similar block counts and long chains start early.
//
// Per block a lane issues two compressions: (IV; h_{j-1} || T_j[0..7]) and
// (state; T_j[8..15] || padding of a 96-byte message).  Three cases leave
// that pattern and take the "special" path, entered only when some lane of
// the wave needs it:
//   * the first block of an unsalted chain: a 64-byte message T_0, whose
//     second compression is the constant padding block;
//   * the boundary block k > 0: a 128-byte message sigma || h_{k-1} || T_k,
//     three compressions; the first, (IV; sigma || h_{k-1}), runs as an
//     extra step and the usual two then take (T_k) and the padding block;
//   * the root-salted first block needs no special path: it is the usual
//     pattern with sigma in place of h_{-1}.
// The hot path is fully unrolled with the round constants as immediates; the
// special path uses a rolled compression reading them from constant memory,
// which keeps the kernel's code within the instruction cache.
//
// Token ids are little-endian int32 (4 bytes each, no separator); SHA-256
// words are big-endian, so each token word is byte-swapped on load.  Digests
// are stored as their big-endian byte serialisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"
#include "sha256_cdna4.h"

#ifndef KVGOV_PAIR_DEFAULT
#define KVGOV_PAIR_DEFAULT 1
#endif
#ifndef KVGOV_PAIRS
#define KVGOV_PAIRS 1
#endif

namespace kvgov {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4), aligned(4)));

__constant__ Sha256Tables kShaDev = make_tables();

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ void load_raw(const int32_t *p, u32x4 raw[4]) {
  const u32x4 *q = reinterpret_cast<const u32x4 *>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) raw[i] = q[i];
}

__device__ __forceinline__ void swap_block(const u32x4 raw[4], uint32_t T[16]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    T[4 * i + 0] = bswap(raw[i].x);
    T[4 * i + 1] = bswap(raw[i].y);
    T[4 * i + 2] = bswap(raw[i].z);
    T[4 * i + 3] = bswap(raw[i].w);
  }
}

__device__ __forceinline__ void store_digest(uint8_t *dst, const uint32_t H[8]) {
  u32x4 *q = reinterpret_cast<u32x4 *>(dst);
  q[0] = u32x4{bswap(H[0]), bswap(H[1]), bswap(H[2]), bswap(H[3])};
  q[1] = u32x4{bswap(H[4]), bswap(H[5]), bswap(H[6]), bswap(H[7])};
}

__device__ __forceinline__ void load_digest(const uint8_t *src, uint32_t H[8]) {
  const u32x4 *q = reinterpret_cast<const u32x4 *>(src);
  const u32x4 a = q[0], b = q[1];
  H[0] = bswap(a.x); H[1] = bswap(a.y); H[2] = bswap(a.z); H[3] = bswap(a.w);
  H[4] = bswap(b.x); H[5] = bswap(b.y); H[6] = bswap(b.z); H[7] = bswap(b.w);
}

// Compression with the 64 rounds in 4 groups of 16 and the constants read
// from constant memory: same result as compress(), a quarter of the code.
__device__ __forceinline__ void compress_rolled(uint32_t st[8], uint32_t w[16]) {
  uint32_t a = st[0], b = st[1], c = st[2], d = st[3];
  uint32_t e = st[4], f = st[5], g = st[6], h = st[7];
#pragma unroll 1
  for (int grp = 0; grp < 4; ++grp) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (grp > 0) {
        w[i] = small_sigma1(w[(i + 14) & 15]) + w[(i + 9) & 15] +
               small_sigma0(w[(i + 1) & 15]) + w[i];
      }
      const uint32_t t1 = h + big_sigma1(e) + ch(e, f, g) + kShaDev.K[grp * 16 + i] + w[i];
      const uint32_t t2 = big_sigma0(a) + maj(a, b, c);
      h = g; g = f; f = e; e = d + t1;
      d = c; c = b; b = a; a = t1 + t2;
    }
  }
  st[0] += a; st[1] += b; st[2] += c; st[3] += d;
  st[4] += e; st[5] += f; st[6] += g; st[7] += h;
}

// ---------------------------------------------------------------------------
// a1: salts
// ---------------------------------------------------------------------------

struct SaltArgs {
  uint32_t key[16];  // K zero-padded to 64 bytes, as big-endian words
  const uint8_t *ids;
  int32_t id_len;
  int32_t P;
  uint8_t *salts;
};

// sigma_p = H((K ^ opad) || H((K ^ ipad) || id_p))   (RFC 2104 over SHA-256)
__global__ __launch_bounds__(64) void k_salts(SaltArgs a) {
  const int p = blockIdx.x * kWave + threadIdx.x;
  if (p >= a.P) return;
  const uint8_t *id = a.ids + (int64_t)p * a.id_len;
  const int L = a.id_len;
  uint32_t st[8], w[16];
  set_iv(st);
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = a.key[i] ^ 0x36363636u;
  compress(st, w);
  const int nblk = (L + 9 + 63) / 64;  // id, 0x80, 64-bit length
  for (int blk = 0; blk < nblk; ++blk) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      uint32_t word = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int pos = blk * 64 + 4 * i + q;
        const uint32_t byte = pos < L ? (uint32_t)id[pos] : (pos == L ? 0x80u : 0u);
        word = (word << 8) | byte;
      }
      w[i] = word;
    }
    if (blk == nblk - 1) {
      const uint64_t bits = (uint64_t)(64 + L) * 8u;
      w[14] = (uint32_t)(bits >> 32);
      w[15] = (uint32_t)bits;
    }
    compress(st, w);
  }
  uint32_t o[8];
  set_iv(o);
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = a.key[i] ^ 0x5c5c5c5cu;
  compress(o, w);
#pragma unroll
  for (int i = 0; i < 8; ++i) w[i] = st[i];
  w[8] = 0x80000000u;
#pragma unroll
  for (int i = 9; i < 15; ++i) w[i] = 0;
  w[15] = (64 + 32) * 8;
  compress(o, w);
  store_digest(a.salts + (int64_t)p * 32, o);
}

// ---------------------------------------------------------------------------
// output layout: blk_offsets = exclusive prefix sum of len // 16
// ---------------------------------------------------------------------------

constexpr int kScanThreads = 256;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanThreads * kScanItems;

__device__ __forceinline__ int64_t req_blocks(const int64_t *tok_offsets, int64_t r,
                                              int32_t *status) {
  const int64_t len = tok_offsets[r + 1] - tok_offsets[r];
  if (len < 0) {
    latch(status, KVGOV_E_OFFSETS);
    return 0;
  }
  return len >> 4;
}

// inclusive scan across the 256 threads of a workgroup
__device__ __forceinline__ int64_t block_inclusive_scan(int64_t v, int64_t *lds_waves) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t u = __shfl_up(v, d, 64);
    if (lane >= d) v += u;
  }
  if (lane == 63) lds_waves[wid] = v;
  __syncthreads();
  int64_t before = 0;
  for (int i = 0; i < wid; ++i) before += lds_waves[i];
  __syncthreads();
  return v + before;
}

__global__ __launch_bounds__(kScanThreads) void k_blk_partial(const int64_t *tok_offsets,
                                                              int32_t n, int64_t *partial,
                                                              int32_t *status) {
  __shared__ int64_t lds[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t r = base + (int64_t)i * kScanThreads + threadIdx.x;
    if (r < n) s += req_blocks(tok_offsets, r, status);
  }
  const int64_t inc = block_inclusive_scan(s, lds);
  if (threadIdx.x == kScanThreads - 1) partial[blockIdx.x] = inc;
}

// single workgroup: exclusive scan of the tile sums, in place
__global__ __launch_bounds__(kScanThreads) void k_blk_scan_partials(int64_t *partial,
                                                                    int64_t count) {
  __shared__ int64_t lds[kScanThreads / 64];
  __shared__ int64_t chunk_total;
  int64_t carry = 0;
  for (int64_t base = 0; base < count; base += kScanThreads) {
    const int64_t i = base + threadIdx.x;
    const int64_t v = i < count ? partial[i] : 0;
    const int64_t inc = block_inclusive_scan(v, lds);
    if (i < count) partial[i] = carry + inc - v;
    if (threadIdx.x == kScanThreads - 1) chunk_total = inc;
    __syncthreads();
    carry += chunk_total;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kScanThreads) void k_blk_write(const int64_t *tok_offsets, int32_t n,
                                                            const int64_t *partial,
                                                            int64_t *blk_offsets,
                                                            int32_t *status) {
  __shared__ int64_t lds[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  // each thread owns kScanItems consecutive requests
  const int64_t r0 = base + (int64_t)threadIdx.x * kScanItems;
  int64_t c[kScanItems];
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t r = r0 + i;
    c[i] = r < n ? req_blocks(tok_offsets, r, status) : 0;
    s += c[i];
  }
  const int64_t inc = block_inclusive_scan(s, lds);
  int64_t run = partial[blockIdx.x] + inc - s;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t r = r0 + i;
    if (r < n) blk_offsets[r] = run;
    run += c[i];
    if (r == n - 1) blk_offsets[n] = run;
  }
  if (n == 0 && blockIdx.x == 0 && threadIdx.x == 0) blk_offsets[0] = 0;
}

// ---------------------------------------------------------------------------
// longest-first ordering: counting sort of requests by block count
// ---------------------------------------------------------------------------

constexpr int kOrderBuckets = 4096;  // block counts >= 4095 share the top bucket

__device__ __forceinline__ int order_bucket(const int64_t *tok_offsets, int32_t r) {
  const int64_t len = tok_offsets[r + 1] - tok_offsets[r];
  const int64_t nb = len > 0 ? (len >> 4) : 0;
  return (int)(nb < kOrderBuckets - 1 ? nb : kOrderBuckets - 1);
}

// Histogram and scatter work on tiles of kOrderTile requests per workgroup and
// count in LDS first, so global atomics are one per (tile, non-empty bucket):
// per-request atomics on a few hot bucket counters serialise (4 ms for a
// 1.25M-request batch).
constexpr int kOrderThreads = 1024;
constexpr int kOrderPerThread = 4;
constexpr int64_t kOrderTile = (int64_t)kOrderThreads * kOrderPerThread;

__global__ __launch_bounds__(kOrderThreads) void k_order_hist(const int64_t *tok_offsets,
                                                              int32_t n, int32_t *hist) {
  __shared__ int32_t h[kOrderBuckets];
  for (int i = threadIdx.x; i < kOrderBuckets; i += kOrderThreads) h[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kOrderTile;
#pragma unroll
  for (int k = 0; k < kOrderPerThread; ++k) {
    const int64_t r = base + (int64_t)k * kOrderThreads + threadIdx.x;
    if (r < n) atomicAdd(&h[order_bucket(tok_offsets, (int32_t)r)], 1);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kOrderBuckets; i += kOrderThreads)
    if (h[i]) atomicAdd(&hist[i], h[i]);
}

// one workgroup: start[b] = number of requests in buckets above b (descending order)
__global__ __launch_bounds__(256) void k_order_scan(int32_t *hist) {
  __shared__ int32_t sums[256];
  constexpr int per = kOrderBuckets / 256;
  const int t = threadIdx.x;
  // thread t owns buckets kOrderBuckets-1-t*per down to kOrderBuckets-(t+1)*per,
  // so the highest buckets go to thread 0
  int32_t local = 0;
  for (int i = 0; i < per; ++i) local += hist[kOrderBuckets - 1 - (t * per + i)];
  sums[t] = local;
  __syncthreads();
  int32_t before = 0;
  for (int i = 0; i < t; ++i) before += sums[i];
  __syncthreads();
  for (int i = 0; i < per; ++i) {
    const int b = kOrderBuckets - 1 - (t * per + i);
    const int32_t cnt = hist[b];
    hist[b] = before;
    before += cnt;
  }
}

__global__ __launch_bounds__(kOrderThreads) void k_order_scatter(const int64_t *tok_offsets,
                                                                 int32_t n, int32_t *cursor,
                                                                 int32_t *order) {
  __shared__ int32_t cnt[kOrderBuckets];
  __shared__ int32_t at[kOrderBuckets];
  for (int i = threadIdx.x; i < kOrderBuckets; i += kOrderThreads) cnt[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kOrderTile;
  int32_t bucket[kOrderPerThread], rank[kOrderPerThread];
#pragma unroll
  for (int k = 0; k < kOrderPerThread; ++k) {
    const int64_t r = base + (int64_t)k * kOrderThreads + threadIdx.x;
    bucket[k] = -1;
    if (r < n) {
      bucket[k] = order_bucket(tok_offsets, (int32_t)r);
      rank[k] = atomicAdd(&cnt[bucket[k]], 1);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kOrderBuckets; i += kOrderThreads)
    if (cnt[i]) at[i] = atomicAdd(&cursor[i], cnt[i]);
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kOrderPerThread; ++k) {
    if (bucket[k] >= 0) {
      const int64_t r = base + (int64_t)k * kOrderThreads + threadIdx.x;
      order[at[bucket[k]] + rank[k]] = (int32_t)r;
    }
  }
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t *p, int64_t count, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) p[i] = v;
}

// ---------------------------------------------------------------------------
// a2/a3: chains
// ---------------------------------------------------------------------------

struct ChainArgs {
  const int32_t *tokens;
  int64_t n_tokens;
  const int64_t *tok_offsets;
  const int64_t *blk_offsets;
  const int32_t *principal;
  const uint8_t *salts;
  int32_t P;
  int32_t n;
  const int32_t *boundary_tok;
  uint8_t *hashes;
  int64_t n_blocks;
  const int32_t *order;  // NULL: request i on lane i
  int32_t *status;
};

// Per-request set-up shared by both chain kernels.  Returns false (after
// latching the error) for a request that must write nothing.
struct ChainReq {
  const int32_t *tp;  // first token
  uint8_t *out;       // first output row
  int64_t nf;         // full blocks
  int64_t k;          // salted block (boundary mode), else -1
  uint32_t sig[8];    // salt as state words (salted modes)
  bool salted_root;   // first block carries the salt (root, or boundary k = 0)
};

template <int MODE>
__device__ __forceinline__ bool chain_setup(const ChainArgs &a, int32_t r, ChainReq &q) {
  const int64_t t0 = a.tok_offsets[r], t1 = a.tok_offsets[r + 1];
  if (t0 < 0 || t1 < t0 || t1 > a.n_tokens) {
    latch(a.status, KVGOV_E_OFFSETS);
    return false;
  }
  const int64_t len = t1 - t0;
  q.nf = len >> 4;
  const int64_t b0 = a.blk_offsets[r];
  if (b0 < 0 || a.blk_offsets[r + 1] - b0 != q.nf || b0 + q.nf > a.n_blocks) {
    latch(a.status, KVGOV_E_OFFSETS);
    return false;
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) q.sig[i] = 0;
  if (MODE != KVGOV_NONE) {
    const int32_t p = a.principal[r];
    if (p < 0 || p >= a.P) {
      latch(a.status, KVGOV_E_PRINCIPAL);
      return false;
    }
    load_digest(a.salts + (int64_t)p * 32, q.sig);
  }
  q.k = -1;
  if (MODE == KVGOV_BOUNDARY) {
    const int32_t bt = a.boundary_tok[r];
    if (bt < 0 || bt > len) {
      latch(a.status, KVGOV_E_BOUNDARY);
      return false;
    }
    q.k = bt >> 4;
  }
  q.tp = a.tokens + t0;
  q.out = a.hashes + b0 * 32;
  q.salted_root = (MODE == KVGOV_ROOT) || (MODE == KVGOV_BOUNDARY && q.k == 0);
  return true;
}

// The special path, per lane (rolled compressions):
//   normal  : (IV; h || T[0..7])        (state; T[8..15] || pad96)
//   u0      : (IV; T[0..15])            (state; pad64)
//   boundary: (IV; sigma || h) -> X,   (X; T[0..15])   (state; pad128)
// H (h_{j-1} in, h_j out) and the block's token words T.
__device__ __forceinline__ void special_block(uint32_t H[8], const uint32_t T[16],
                                              const uint32_t sig[8], bool u0, bool bnd) {
  uint32_t X[8], st[8], w[16];
  set_iv(X);
  if (bnd) {
#pragma unroll
    for (int q = 0; q < 8; ++q) { w[q] = sig[q]; w[8 + q] = H[q]; }
    compress_rolled(X, w);
  }
  const bool whole = u0 || bnd;  // first compression takes all 16 token words
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    st[q] = X[q];
    w[q] = whole ? T[q] : H[q];
    w[8 + q] = whole ? T[8 + q] : T[q];
  }
  compress_rolled(st, w);
#pragma unroll
  for (int q = 0; q < 8; ++q) w[q] = whole ? (q == 0 ? 0x80000000u : 0u) : T[8 + q];
  w[8] = whole ? 0u : 0x80000000u;
#pragma unroll
  for (int q = 9; q < 15; ++q) w[q] = 0;
  w[15] = u0 ? 64 * 8 : (bnd ? 128 * 8 : 96 * 8);
  compress_rolled(st, w);
#pragma unroll
  for (int q = 0; q < 8; ++q) H[q] = st[q];
}

// Padding words 8..15 of the second block of a 96-byte message.
__device__ __forceinline__ void pad96_tail(uint32_t w[16]) {
  w[8] = 0x80000000u;
#pragma unroll
  for (int q = 9; q < 15; ++q) w[q] = 0;
  w[15] = 96 * 8;
}

// One lane per request.  Every instruction of a compression (rounds and
// message schedule) is issued by the lane's wave.
template <int MODE>
__global__ __launch_bounds__(256) void k_chains(ChainArgs a) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int32_t r = a.order ? a.order[i] : i;
  ChainReq q;
  if (!chain_setup<MODE>(a, r, q) || q.nf == 0) return;
  const int64_t nf = q.nf;

  // H holds h_{j-1} as state words; a root-salted first block (and k == 0 in
  // boundary mode) is the usual pattern with sigma in place of h_{-1}.
  uint32_t H[8];
#pragma unroll
  for (int w = 0; w < 8; ++w) H[w] = q.salted_root ? q.sig[w] : 0u;

  u32x4 nxt[4];
  load_raw(q.tp, nxt);
  const bool plain_first = !q.salted_root;

  for (int64_t j = 0; j < nf; ++j) {
    uint32_t T[16];
    swap_block(nxt, T);
    if (j + 1 < nf) load_raw(q.tp + 16 * (j + 1), nxt);

    const bool u0 = plain_first && j == 0;
    const bool bnd = (MODE == KVGOV_BOUNDARY) && j == q.k && q.k > 0;
    if (MODE == KVGOV_ROOT || !__any(u0 || bnd)) {
      // hot path: (IV; h || T[0..7]) then (state; T[8..15] || pad96)
      uint32_t st[8], w[16];
      set_iv(st);
#pragma unroll
      for (int x = 0; x < 8; ++x) { w[x] = H[x]; w[8 + x] = T[x]; }
      compress(st, w);
#pragma unroll
      for (int x = 0; x < 8; ++x) w[x] = T[8 + x];
      pad96_tail(w);
      compress(st, w);
#pragma unroll
      for (int x = 0; x < 8; ++x) H[x] = st[x];
    } else {
      special_block(H, T, q.sig, u0, bnd);
    }
    store_digest(q.out + j * 32, H);
  }
}

// ---------------------------------------------------------------------------
// wave-pair chain kernel
// ---------------------------------------------------------------------------
//
// A chain is latency-bound: one wave advances 64 chains at the issue rate of
// its SIMD, and a block costs ~2800 vector instructions, a third of them the
// message schedule.  The schedule does not feed back into the rounds except
// through its output words, so a second wave on another SIMD computes it and
// hands the words over through LDS:
//   wave 0 ("rounds")   : the 64 rounds of each compression, state in registers;
//   wave 1 ("schedule") : W[16..63] of both compressions of every block.
// Lane l of both waves owns the same request.  Per block j:
//   phase 1  rounds: C1 rounds 0-15 (message h_{j-1} || T[0..7] in registers)
//            schedule: reads h_{j-1} from LDS, computes C1's W[16..31]
//   phase 2  rounds: C1 rounds 16-31       schedule: C1's W[32..47]
//   phase 3  rounds: C1 rounds 32-47       schedule: C1's W[48..63]
//   phase 4  rounds: C1 rounds 48-63, then all of C2 (its W[16..63] were
//            computed during block j-1: the C2 message T[8..15] || padding
//            depends on tokens only); writes h_j to LDS and the digest
//            schedule: C2's W[16..63] of block j+1 (double buffered)
// with a workgroup barrier after each phase.  Iterations where a lane of the
// wave has a special block (unsalted first block, boundary block) run the
// special path entirely on the rounds wave; the schedule wave then only
// prepares the next block's C2 words.  Both waves derive every branch and
// trip count from the same per-lane data, so they meet the same barriers.

struct PairLds {
  uint32_t h[8][kWave];          // h_{j-1} per lane
  uint32_t w1[48][kWave];        // C1's W[16..63]
  uint32_t w2[2][48][kWave];     // C2's W[16..63], double buffered by block parity
};

struct Sha8 {
  uint32_t a, b, c, d, e, f, g, h;
};

__device__ __forceinline__ void round_w(Sha8 &s, uint32_t kt, uint32_t w) {
  const uint32_t t1 = s.h + big_sigma1(s.e) + ch(s.e, s.f, s.g) + kt + w;
  const uint32_t t2 = big_sigma0(s.a) + maj(s.a, s.b, s.c);
  s.h = s.g; s.g = s.f; s.f = s.e; s.e = s.d + t1;
  s.d = s.c; s.c = s.b; s.b = s.a; s.a = t1 + t2;
}

__device__ __forceinline__ Sha8 sha8_iv() {
  return Sha8{kSha.H0[0], kSha.H0[1], kSha.H0[2], kSha.H0[3],
              kSha.H0[4], kSha.H0[5], kSha.H0[6], kSha.H0[7]};
}

__device__ __forceinline__ Sha8 sha8_load(const uint32_t st[8]) {
  return Sha8{st[0], st[1], st[2], st[3], st[4], st[5], st[6], st[7]};
}

__device__ __forceinline__ void sha8_add(uint32_t st[8], const Sha8 &s) {
  st[0] += s.a; st[1] += s.b; st[2] += s.c; st[3] += s.d;
  st[4] += s.e; st[5] += s.f; st[6] += s.g; st[7] += s.h;
}

// 16 schedule words from LDS into registers
__device__ __forceinline__ void load16(uint32_t w[16], const uint32_t (*wl)[kWave], int base,
                                       int lane) {
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = wl[base + i][lane];
}

// rounds t0..t0+11 and t0..t0+3 with W[t0 + i] = w[i]
__device__ __forceinline__ void rounds12(Sha8 &s, const uint32_t *w, int t0) {
#pragma unroll
  for (int i = 0; i < 12; ++i) round_w(s, kSha.K[t0 + i], w[i]);
}
__device__ __forceinline__ void rounds4(Sha8 &s, const uint32_t *w, int t0) {
#pragma unroll
  for (int i = 0; i < 4; ++i) round_w(s, kSha.K[t0 + i], w[i]);
}

// 16 schedule words W[t..t+15] from the rolling window w (W[t-16..t-1]),
// stored to out[base + i][lane]
__device__ __forceinline__ void sched16(uint32_t w[16], uint32_t (*out)[kWave], int base,
                                        int lane) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    w[i] = small_sigma1(w[(i + 14) & 15]) + w[(i + 9) & 15] + small_sigma0(w[(i + 1) & 15]) +
           w[i];
    out[base + i][lane] = w[i];
  }
}

// Block-count summary of a request used to keep the waves of a workgroup in
// lockstep: every wave evaluates it for every pair's request of its lane.
struct PairPeek {
  int64_t nf;
  int64_t k;
  bool plain_first;
};

template <int MODE>
__device__ __forceinline__ PairPeek pair_peek(const ChainArgs &a, int32_t i) {
  PairPeek p{0, -1, false};
  if (i < a.n) {
    ChainReq q;
    const int32_t r = a.order ? a.order[i] : i;
    if (chain_setup<MODE>(a, r, q)) p = PairPeek{q.nf, q.k, !q.salted_root};
  }
  return p;
}

template <int MODE>
__device__ __forceinline__ bool pair_special(const PairPeek &p, int64_t j) {
  const bool act = j < p.nf;
  return act && ((p.plain_first && j == 0) ||
                 ((MODE == KVGOV_BOUNDARY) && j == p.k && p.k > 0));
}

// PAIRS wave pairs per workgroup: waves 2p (rounds) and 2p+1 (schedule) of
// pair p own the 64 requests blockIdx.x * 64 * PAIRS + 64 p + lane.  Trip
// count and special iterations are decided over all pairs of the workgroup,
// so every wave meets every barrier.
template <int MODE, int PAIRS>
__global__ __launch_bounds__(2 * PAIRS * kWave) void k_chains_pair(ChainArgs a) {
  __shared__ PairLds Lp[PAIRS];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int pair = wave >> 1;
  const bool rounds_wave = (wave & 1) == 0;
  PairLds &L = Lp[pair];
  const int32_t base = blockIdx.x * kWave * PAIRS;
  const int32_t i = base + pair * kWave + lane;

  // identical set-up on both waves of a pair; a rejected or empty request
  // has nf = 0 (both waves latch the same error, the first one wins)
  ChainReq q;
  bool ok = false;
  if (i < a.n) {
    const int32_t r = a.order ? a.order[i] : i;
    ok = chain_setup<MODE>(a, r, q);
  }
  const int64_t nf = ok ? q.nf : 0;
  PairPeek peek[PAIRS];
#pragma unroll
  for (int p = 0; p < PAIRS; ++p)
    peek[p] = (p == pair) ? PairPeek{nf, ok ? q.k : -1, ok && !q.salted_root}
                          : pair_peek<MODE>(a, base + p * kWave + lane);
  // workgroup-uniform trip count
  int64_t J = 0;
#pragma unroll
  for (int p = 0; p < PAIRS; ++p) J = peek[p].nf > J ? peek[p].nf : J;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    const int64_t o = __shfl_xor(J, d, kWave);
    J = o > J ? o : J;
  }
  const bool plain_first = ok && !q.salted_root;

  uint32_t H[8];
#pragma unroll
  for (int w = 0; w < 8; ++w) H[w] = (ok && q.salted_root) ? q.sig[w] : 0u;

  u32x4 nxt[4];    // tokens of the next block (both waves)
  uint32_t T[16];  // tokens of the current block
  if (nf > 0) load_raw(q.tp, nxt);

  // prologue: h_{-1} to LDS; the schedule wave prepares C2's words of block 0
  if (rounds_wave) {
#pragma unroll
    for (int w = 0; w < 8; ++w) L.h[w][lane] = H[w];
  } else if (nf > 0) {
    uint32_t T0[16];
    swap_block(nxt, T0);
    uint32_t w[16];
#pragma unroll
    for (int x = 0; x < 8; ++x) w[x] = T0[8 + x];
    pad96_tail(w);
    sched16(w, L.w2[0], 0, lane);
    sched16(w, L.w2[0], 16, lane);
    sched16(w, L.w2[0], 32, lane);
  }
  __syncthreads();

  for (int64_t j = 0; j < J; ++j) {
    const bool act = j < nf;
    if (act) {
      swap_block(nxt, T);
      if (j + 1 < nf) load_raw(q.tp + 16 * (j + 1), nxt);
    }
    const bool u0 = act && plain_first && j == 0;
    const bool bnd = act && (MODE == KVGOV_BOUNDARY) && j == q.k && q.k > 0;
    const int nb = (int)((j + 1) & 1);  // C2 buffer of block j+1
    const bool next = j + 1 < nf;

    bool special_any = false;
    if (MODE != KVGOV_ROOT) {
#pragma unroll
      for (int p = 0; p < PAIRS; ++p) special_any |= pair_special<MODE>(peek[p], j);
    }
    if (MODE != KVGOV_ROOT && __any(special_any)) {
      // special iteration: the rounds wave does the whole block itself
      if (rounds_wave) {
        if (act) {
          special_block(H, T, q.sig, u0, bnd);
#pragma unroll
          for (int w = 0; w < 8; ++w) L.h[w][lane] = H[w];
          store_digest(q.out + j * 32, H);
        }
      } else if (next) {
        uint32_t Tn[16], w[16];
        swap_block(nxt, Tn);
#pragma unroll
        for (int x = 0; x < 8; ++x) w[x] = Tn[8 + x];
        pad96_tail(w);
        sched16(w, L.w2[nb], 0, lane);
        sched16(w, L.w2[nb], 16, lane);
        sched16(w, L.w2[nb], 32, lane);
      }
      __syncthreads();
      continue;
    }

    if (rounds_wave) {
      // Each barrier sits 4 rounds before the words it releases are needed,
      // so the LDS reads issued right after it overlap those 4 rounds; the
      // scheduling barriers keep the compiler from sinking the reads to
      // their uses.  C2's words (written during the previous block) are read
      // one group ahead.
      Sha8 s = sha8_iv();
      uint32_t wa[16], wb[16];
      if (act) {
#pragma unroll
        for (int t = 0; t < 8; ++t) round_w(s, kSha.K[t], H[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) round_w(s, kSha.K[8 + t], T[t]);
      }
      __syncthreads();  // C1 W[16..31] ready
      if (act) {
        load16(wa, L.w1, 0, lane);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 4; t < 8; ++t) round_w(s, kSha.K[8 + t], T[t]);
        rounds12(s, wa, 16);
      }
      __syncthreads();  // C1 W[32..47] ready
      if (act) {
        load16(wb, L.w1, 16, lane);
        __builtin_amdgcn_sched_barrier(0);
        rounds4(s, wa + 12, 28);
        rounds12(s, wb, 32);
      }
      __syncthreads();  // C1 W[48..63] ready
      if (act) {
        const uint32_t(*w2)[kWave] = L.w2[j & 1];
        load16(wa, L.w1, 32, lane);
        __builtin_amdgcn_sched_barrier(0);
        rounds4(s, wb + 12, 44);
        load16(wb, w2, 0, lane);  // C2 W[16..31]
        __builtin_amdgcn_sched_barrier(0);
        rounds12(s, wa, 48);
        rounds4(s, wa + 12, 60);
        uint32_t st[8];
#pragma unroll
        for (int w = 0; w < 8; ++w) st[w] = kSha.H0[w];
        sha8_add(st, s);
        // C2: rounds 0-15 from registers (T[8..15] || pad96), 16-63 from LDS
        Sha8 s2 = sha8_load(st);
        load16(wa, w2, 16, lane);  // C2 W[32..47]
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < 8; ++t) round_w(s2, kSha.K[t], T[8 + t]);
        round_w(s2, kSha.K[8], 0x80000000u);
#pragma unroll
        for (int t = 9; t < 15; ++t) round_w(s2, kSha.K[t], 0u);
        round_w(s2, kSha.K[15], 96 * 8);
        rounds12(s2, wb, 16);
        rounds4(s2, wb + 12, 28);
        load16(wb, w2, 32, lane);  // C2 W[48..63]
        __builtin_amdgcn_sched_barrier(0);
        rounds12(s2, wa, 32);
        rounds4(s2, wa + 12, 44);
        rounds12(s2, wb, 48);
        rounds4(s2, wb + 12, 60);
        sha8_add(st, s2);
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          H[w] = st[w];
          L.h[w][lane] = st[w];
        }
        store_digest(q.out + j * 32, H);
      }
      __syncthreads();
    } else {
      // ---- schedule wave
      uint32_t w[16];
      if (act) {
#pragma unroll
        for (int x = 0; x < 8; ++x) { w[x] = L.h[x][lane]; w[8 + x] = T[x]; }
        sched16(w, L.w1, 0, lane);
      }
      __syncthreads();
      if (act) sched16(w, L.w1, 16, lane);
      __syncthreads();
      if (act) sched16(w, L.w1, 32, lane);
      __syncthreads();
      if (next) {
        uint32_t Tn[16];
        swap_block(nxt, Tn);
#pragma unroll
        for (int x = 0; x < 8; ++x) w[x] = Tn[8 + x];
        pad96_tail(w);
        sched16(w, L.w2[nb], 0, lane);
        sched16(w, L.w2[nb], 16, lane);
        sched16(w, L.w2[nb], 32, lane);
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

// Dynamic LDS per chain workgroup: just over half a CU's LDS.
static size_t chain_lds_reserve() {
  static std::mutex mu;
  static std::vector<size_t> per_dev;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 96 * 1024;
  std::lock_guard<std::mutex> g(mu);
  if ((int)per_dev.size() <= dev) per_dev.resize(dev + 1, 0);
  if (per_dev[dev] == 0) {
    int cu_lds = 0, blk_lds = 0;
    if (hipDeviceGetAttribute(&cu_lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
            hipSuccess || cu_lds <= 0)
      cu_lds = 160 * 1024;
    if (hipDeviceGetAttribute(&blk_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
            hipSuccess || blk_lds <= 0)
      blk_lds = cu_lds;
    per_dev[dev] = std::min<size_t>((size_t)cu_lds / 2 + 4096, (size_t)blk_lds);
  }
  return per_dev[dev];
}

static int cu_lds_bytes() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
          hipSuccess ||
      v <= 0)
    v = 160 * 1024;
  return v;
}

// Dynamic LDS of a wave-pair workgroup so that at most `per_cu` pair
// workgroups share a CU (1: more than half of the CU's LDS; 2: more than a
// third, at most half).
static size_t pair_lds_reserve(int per_cu) {
  const size_t cu = (size_t)cu_lds_bytes();
  const size_t want = per_cu == 1 ? cu / 2 + 4096 : cu / 2 - 1024;
  const size_t fixed = KVGOV_PAIRS * sizeof(PairLds);
  return want > fixed ? want - fixed : 0;
}

// Pair workgroups per CU for a batch of n requests: the wave-pair kernel
// shortens every chain but needs two waves per 64 requests, so it runs while
// the batch fits in one or two pairs per CU (latency-bound batches); larger
// batches keep every SIMD busy with the single-wave kernel (0).
static int pair_slots(int32_t n) {
  if (!KVGOV_PAIR_DEFAULT || n <= 0) return 0;
  const int64_t pairs = ceil_div(n, (int64_t)kWave * KVGOV_PAIRS);
  const int64_t cus = device_cu_count();
  if (pairs <= cus) return 1;
  if (pairs <= 2 * cus) return 2;
  return 0;
}

int device_cu_count() {
  static std::mutex mu;
  static std::vector<int> cus;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> g(mu);
  if ((int)cus.size() <= dev) cus.resize(dev + 1, 0);
  if (cus[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v <= 0)
      v = 256;
    cus[dev] = v;
  }
  return cus[dev];
}

}  // namespace kvgov

using namespace kvgov;

extern "C" {

const char *kvgov_strerror(int code) {
  switch (code) {
    case KVGOV_OK: return "ok";
    case KVGOV_E_INVAL: return "invalid argument";
    case KVGOV_E_UNSUPPORTED: return "unsupported argument (block size 16 and keys up to 64 bytes)";
    case KVGOV_E_OFFSETS: return "offsets not monotone, out of bounds, or not matching len // 16";
    case KVGOV_E_BOUNDARY: return "boundary_tok outside [0, len]";
    case KVGOV_E_PRINCIPAL: return "principal index outside [0, P)";
    case KVGOV_E_FULL: return "cache table full";
    case KVGOV_E_HIP: return "HIP runtime error";
    case KVGOV_E_NOMEM: return "device allocation failed";
    case KVGOV_E_CAPACITY: return "export buffer too small";
    case KVGOV_E_DEVICE: return "cache used with a different current device";
    case KVGOV_E_INTERNAL: return "bounded wait exhausted inside a kernel";
    default: return "unknown error code";
  }
}

int kvgov_version(void) { return (1 << 16) | 0; }

int kvgov_salts(const uint8_t *K, size_t K_len, const uint8_t *principal_ids, int32_t id_len,
                int32_t P, uint8_t *salts, void *stream) {
  if (!K || K_len == 0 || P < 0 || id_len < 0 || id_len > KVGOV_MAX_ID_BYTES)
    return KVGOV_E_INVAL;
  if (K_len > KVGOV_MAX_KEY_BYTES) return KVGOV_E_UNSUPPORTED;
  if (P > 0 && (!salts || (!principal_ids && id_len > 0))) return KVGOV_E_INVAL;
  if (P > 0 && (reinterpret_cast<uintptr_t>(salts) & 3)) return KVGOV_E_INVAL;
  if (P == 0) return KVGOV_OK;
  SaltArgs a{};
  for (size_t i = 0; i < K_len; ++i) a.key[i / 4] |= (uint32_t)K[i] << (24 - 8 * (i % 4));
  a.ids = principal_ids;
  a.id_len = id_len;
  a.P = P;
  a.salts = salts;
  hipLaunchKernelGGL(k_salts, dim3((unsigned)ceil_div(P, kWave)), dim3(kWave), 0,
                     as_stream(stream), a);
  const int rc = launch_status();
  volatile uint32_t *wipe = a.key;  // the kernel argument was copied at launch
  for (int i = 0; i < 16; ++i) wipe[i] = 0;
  return rc;
}

int kvgov_block_offsets(const int64_t *tok_offsets, int32_t n, int32_t block_size,
                        int64_t *blk_offsets, int32_t *status, void *stream) {
  if (!tok_offsets || !blk_offsets || !status || n < 0) return KVGOV_E_INVAL;
  if (block_size != KVGOV_BLOCK_SIZE) return KVGOV_E_UNSUPPORTED;
  hipStream_t s = as_stream(stream);
  const int64_t tiles = std::max<int64_t>(1, ceil_div(n, kScanTile));
  int64_t *partial = nullptr;
  if (hipMallocAsync(reinterpret_cast<void **>(&partial), tiles * sizeof(int64_t), s) !=
      hipSuccess)
    return KVGOV_E_NOMEM;
  hipLaunchKernelGGL(k_blk_partial, dim3((unsigned)tiles), dim3(kScanThreads), 0, s,
                     tok_offsets, n, partial, status);
  hipLaunchKernelGGL(k_blk_scan_partials, dim3(1), dim3(kScanThreads), 0, s, partial, tiles);
  hipLaunchKernelGGL(k_blk_write, dim3((unsigned)tiles), dim3(kScanThreads), 0, s, tok_offsets,
                     n, partial, blk_offsets, status);
  int rc = launch_status();
  if (hipFreeAsync(partial, s) != hipSuccess && rc == KVGOV_OK) rc = KVGOV_E_HIP;
  return rc;
}

// Longest-first ordering pays once the batch has about as many waves as the
// chip has SIMDs; below that every wave has a SIMD of its own from the start
// and the kernel takes as long as its longest chain in any order.  (Batches
// that run on the wave-pair kernel are resident all at once and are never
// ordered.)
static int64_t order_min_requests() { return (int64_t)device_cu_count() * 4 * kWave / 2; }

int kvgov_hash_chains(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_offsets,
                      int32_t n, const int32_t *principal, const uint8_t *salts, int32_t P,
                      int32_t mode, const int32_t *boundary_tok, int32_t block_size,
                      const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                      int32_t *status, void *stream) {
  if (n < 0 || n_tokens < 0 || n_blocks < 0 || !status) return KVGOV_E_INVAL;
  if (mode != KVGOV_NONE && mode != KVGOV_ROOT && mode != KVGOV_BOUNDARY) return KVGOV_E_INVAL;
  if (block_size != KVGOV_BLOCK_SIZE) return KVGOV_E_UNSUPPORTED;
  if (n == 0) return KVGOV_OK;
  if (!tok_offsets || !blk_offsets || (n_tokens > 0 && !tokens) || (n_blocks > 0 && !hashes))
    return KVGOV_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(tokens) & 3) || (reinterpret_cast<uintptr_t>(hashes) & 3))
    return KVGOV_E_INVAL;
  if (mode != KVGOV_NONE && (!principal || !salts || P <= 0)) return KVGOV_E_INVAL;
  if (mode == KVGOV_BOUNDARY && !boundary_tok) return KVGOV_E_INVAL;
  hipStream_t s = as_stream(stream);

  ChainArgs a{};
  a.tokens = tokens;
  a.n_tokens = n_tokens;
  a.tok_offsets = tok_offsets;
  a.blk_offsets = blk_offsets;
  a.principal = principal;
  a.salts = salts;
  a.P = P;
  a.n = n;
  a.boundary_tok = boundary_tok;
  a.hashes = hashes;
  a.n_blocks = n_blocks;
  a.status = status;
  a.order = nullptr;

  const int slots = pair_slots(n);
  int32_t *scratch = nullptr;
  if (!slots && n >= order_min_requests()) {
    const size_t bytes = sizeof(int32_t) * ((size_t)kOrderBuckets + (size_t)n);
    if (hipMallocAsync(reinterpret_cast<void **>(&scratch), bytes, s) != hipSuccess)
      return KVGOV_E_NOMEM;
    int32_t *hist = scratch;
    int32_t *order = scratch + kOrderBuckets;
    hipLaunchKernelGGL(k_fill_i32, dim3(kOrderBuckets / 256), dim3(256), 0, s, hist,
                       (int64_t)kOrderBuckets, 0);
    const dim3 tiles((unsigned)ceil_div(n, kOrderTile));
    hipLaunchKernelGGL(k_order_hist, tiles, dim3(kOrderThreads), 0, s, tok_offsets, n, hist);
    hipLaunchKernelGGL(k_order_scan, dim3(1), dim3(256), 0, s, hist);
    hipLaunchKernelGGL(k_order_scatter, tiles, dim3(kOrderThreads), 0, s, tok_offsets, n, hist,
                       order);
    a.order = order;
  }
  // Launch shape.  A chain wave is bound by its SIMD's issue rate, so it
  // should never share a SIMD while others sit idle.  The dispatcher stacks
  // the waves of concurrent launches on the same SIMDs, and the older wave
  // then takes nearly every issue slot, so the workgroups reserve LDS (unused
  // beyond the kernel's own) to bound how many share a CU.
  if (slots) {
    // wave pairs (rounds wave + schedule wave), one or two pairs per CU
    constexpr int P = KVGOV_PAIRS;
    const dim3 grid((unsigned)ceil_div(n, kWave * P)), block(2 * P * kWave);
    const size_t lds = pair_lds_reserve(slots);
    switch (mode) {
      case KVGOV_NONE: hipLaunchKernelGGL((k_chains_pair<KVGOV_NONE, P>), grid, block, lds, s, a); break;
      case KVGOV_ROOT: hipLaunchKernelGGL((k_chains_pair<KVGOV_ROOT, P>), grid, block, lds, s, a); break;
      default: hipLaunchKernelGGL((k_chains_pair<KVGOV_BOUNDARY, P>), grid, block, lds, s, a); break;
    }
  } else {
    // at most one workgroup per CU; batches of at most one wave per CU run
    // one wave per workgroup, larger ones four (one per SIMD)
    const int threads = (int64_t)n <= (int64_t)device_cu_count() * kWave ? kWave : 4 * kWave;
    const dim3 grid((unsigned)ceil_div(n, threads)), block(threads);
    const size_t lds = chain_lds_reserve();
    switch (mode) {
      case KVGOV_NONE: hipLaunchKernelGGL(k_chains<KVGOV_NONE>, grid, block, lds, s, a); break;
      case KVGOV_ROOT: hipLaunchKernelGGL(k_chains<KVGOV_ROOT>, grid, block, lds, s, a); break;
      default: hipLaunchKernelGGL(k_chains<KVGOV_BOUNDARY>, grid, block, lds, s, a); break;
    }
  }
  int rc = launch_status();
  if (scratch && hipFreeAsync(scratch, s) != hipSuccess && rc == KVGOV_OK) rc = KVGOV_E_HIP;
  return rc;
}

}  // extern "C"
