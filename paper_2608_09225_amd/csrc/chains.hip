// Salts (HMAC-SHA256) and chained block hashes on gfx950.
//
// Paper: per-principal salt sigma_p = HMAC_K(principal_id) (Sec. 4.1); block
// hashes chained h_j = H(h_{j-1}, tokens_j) (Sec. 2.1) with the salt at the
// root (Sec. 4.1) or at the divergence boundary k (Sec. 4.2).
//
// Execution model.  A chain is a strict sequence of SHA-256 compressions
// (h_j needs h_{j-1}), so all parallelism comes from the batch.  Two kernels:
//   * k_chains: one lane owns one request and walks its chain (a wave
//     advances 64 chains); for batches that fill every SIMD, ordered longest
//     first (LPT) so that the lanes of a wave carry similar block counts and
//     long chains start early;
//   * k_chains_lp: three waves per 64 requests, two lanes per request for
//     the rounds and a third wave for the message schedule, which shortens
//     every chain; for batches of at most two workgroups per CU.
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
#include <map>
#include <mutex>
#include <thread>
#include <tuple>
#include <vector>

#include "common.h"
#include "sha256_cdna4.h"

#ifndef KVGOV_LP_COVER
#define KVGOV_LP_COVER 2  // lane-pair kernel: steps between a barrier and its first word
#endif
#ifndef KVGOV_LP_GROUPS
#define KVGOV_LP_GROUPS 16, 32, 48, 64  // lane-pair kernel: schedule group bounds
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

// Token prefetch.  T <- the block held in raw (block j), then raw <- block
// j + 1 (block j again when j is the last, so that the load is
// unconditional).  The scheduling barriers pin the load right after the last
// read of raw: it then writes raw's registers in place, and its latency hides
// behind a block's compressions.  (Issued before those reads, or under a
// condition, the load lands in temporaries that are copied into raw at once,
// which waits for it.)  Callers take the next block before storing the
// current digest: a wait for the load must not also wait for a store issued
// after it.
__device__ __forceinline__ void swap_block(const u32x4 raw[4], uint32_t T[16]);
__device__ __forceinline__ void take_block(u32x4 raw[4], uint32_t T[16], const int32_t *tp,
                                           int64_t j, int64_t nf) {
  swap_block(raw, T);
  __builtin_amdgcn_sched_barrier(0);
  load_raw(tp + 16 * (j + 1 < nf ? j + 1 : j), raw);
  __builtin_amdgcn_sched_barrier(0);
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
// output layout: blk_offsets = exclusive prefix sum of len // 16 (minus the
// start block when resuming)
// ---------------------------------------------------------------------------

constexpr int kScanThreads = 256;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanThreads * kScanItems;

// blocks hashed for request r: full blocks from start[r] on (start NULL: 0)
__device__ __forceinline__ int64_t req_blocks(const int64_t *tok_offsets, const int32_t *start,
                                              int64_t r, int32_t *status) {
  const int64_t len = tok_offsets[r + 1] - tok_offsets[r];
  const int64_t j0 = start ? start[r] : 0;
  if (len < 0 || j0 < 0 || j0 > (len >> 4)) {
    latch(status, KVGOV_E_OFFSETS);
    return 0;
  }
  return (len >> 4) - j0;
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
                                                              const int32_t *start, int32_t n,
                                                              int64_t *partial,
                                                              int32_t *status) {
  __shared__ int64_t lds[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t r = base + (int64_t)i * kScanThreads + threadIdx.x;
    if (r < n) s += req_blocks(tok_offsets, start, r, status);
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

__global__ __launch_bounds__(kScanThreads) void k_blk_write(const int64_t *tok_offsets,
                                                            const int32_t *start, int32_t n,
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
    c[i] = r < n ? req_blocks(tok_offsets, start, r, status) : 0;
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

// bucket of request r: the blocks it hashes, from the block offsets (any
// values are safe here; the chain kernels validate them)
__device__ __forceinline__ int order_bucket(const int64_t *blk_offsets, int32_t r) {
  const int64_t d = blk_offsets[r + 1] - blk_offsets[r];
  const int64_t nb = d > 0 ? d : 0;
  return (int)(nb < kOrderBuckets - 1 ? nb : kOrderBuckets - 1);
}

// Histogram and scatter work on tiles of kOrderTile requests per workgroup and
// count in LDS first, so global atomics are one per (tile, non-empty bucket):
// per-request atomics on a few hot bucket counters serialise (4 ms for a
// 1.25M-request batch).  Workgroups of four waves find room on a busy chip
// (other streams' kernels in flight) far sooner than workgroups of sixteen.
constexpr int kOrderThreads = 256;
constexpr int kOrderPerThread = 16;
constexpr int64_t kOrderTile = (int64_t)kOrderThreads * kOrderPerThread;

__global__ __launch_bounds__(kOrderThreads) void k_order_hist(const int64_t *blk_offsets,
                                                              int32_t n, int32_t *hist) {
  __shared__ int32_t h[kOrderBuckets];
  for (int i = threadIdx.x; i < kOrderBuckets; i += kOrderThreads) h[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kOrderTile;
#pragma unroll
  for (int k = 0; k < kOrderPerThread; ++k) {
    const int64_t r = base + (int64_t)k * kOrderThreads + threadIdx.x;
    if (r < n) atomicAdd(&h[order_bucket(blk_offsets, (int32_t)r)], 1);
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

__global__ __launch_bounds__(kOrderThreads) void k_order_scatter(const int64_t *blk_offsets,
                                                                 int32_t n, int32_t *cursor,
                                                                 int32_t *order,
                                                                 int32_t *status) {
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
      bucket[k] = order_bucket(blk_offsets, (int32_t)r);
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
      // the positions are 0 .. n-1 while the histogram is the batch's own
      const int32_t pos = at[bucket[k]] + rank[k];
      if ((uint32_t)pos < (uint32_t)n)
        order[pos] = (int32_t)r;
      else
        latch(status, KVGOV_E_INTERNAL);
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
  // chain extension: request r resumes at block start[r] from the parent
  // digest parents[r] (NULL: every chain starts at block 0)
  const int32_t *start;
  const uint8_t *parents;
};

// Per-request set-up shared by both chain kernels.  Returns false (after
// latching the error) for a request that must write nothing.
struct ChainReq {
  const int32_t *tp;  // tokens of the first block hashed
  uint8_t *out;       // its output row
  int64_t nf;         // blocks to hash (full blocks from the start block on)
  int64_t j0;         // the start block (0 unless resuming)
  int64_t k;          // salted block (boundary mode), else -1
  int64_t kr;         // iteration (block kr + j0) of a boundary block still to
                      // hash with sigma || h, else -1
  uint32_t sig[8];    // salt as state words (salted modes)
  bool salted_root;   // block 0 carries the salt (root, or boundary k = 0)
};

template <int MODE>
__device__ __forceinline__ bool chain_setup(const ChainArgs &a, int32_t r, ChainReq &q) {
  // r comes from the ordering scratch when the batch is ordered: a value
  // outside the batch would mean that scratch was overwritten
  if ((uint32_t)r >= (uint32_t)a.n) {
    latch(a.status, KVGOV_E_INTERNAL);
    return false;
  }
  const int64_t t0 = a.tok_offsets[r], t1 = a.tok_offsets[r + 1];
  if (t0 < 0 || t1 < t0 || t1 > a.n_tokens) {
    latch(a.status, KVGOV_E_OFFSETS);
    return false;
  }
  const int64_t len = t1 - t0;
  const int64_t full = len >> 4;
  q.j0 = a.start ? a.start[r] : 0;
  if (q.j0 < 0 || q.j0 > full) {
    latch(a.status, KVGOV_E_OFFSETS);
    return false;
  }
  q.nf = full - q.j0;
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
  q.tp = a.tokens + t0 + 16 * q.j0;
  q.out = a.hashes + b0 * 32;
  q.salted_root = (MODE == KVGOV_ROOT) || (MODE == KVGOV_BOUNDARY && q.k == 0);
  q.kr = q.k > 0 && q.k >= q.j0 ? q.k - q.j0 : -1;
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
__device__ __forceinline__ void single_chain(const ChainArgs &a, int32_t i) {
  if (i >= a.n) return;
  const int32_t r = a.order ? a.order[i] : i;
  ChainReq q;
  if (!chain_setup<MODE>(a, r, q) || q.nf == 0) return;
  const int64_t nf = q.nf;

  // H holds h_{j-1} as state words: the parent digest when resuming; a
  // root-salted first block (and k == 0 in boundary mode) is the usual
  // pattern with sigma in place of h_{-1}.
  uint32_t H[8];
  if (q.j0 > 0) {
    load_digest(a.parents + (int64_t)r * 32, H);
  } else {
#pragma unroll
    for (int w = 0; w < 8; ++w) H[w] = q.salted_root ? q.sig[w] : 0u;
  }

  u32x4 nxt[4];
  uint32_t T[16];  // tokens of block j
  load_raw(q.tp, nxt);
  take_block(nxt, T, q.tp, 0, nf);
  const bool plain_first = !q.salted_root && q.j0 == 0;

  // iteration j hashes block q.j0 + j of the chain
  for (int64_t j = 0; j < nf; ++j) {
    const bool u0 = plain_first && j == 0;
    const bool bnd = (MODE == KVGOV_BOUNDARY) && j == q.kr;
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
    // the next block's tokens before the digest store (see take_block)
    take_block(nxt, T, q.tp, j + 1 < nf ? j + 1 : j, nf);
    store_digest(q.out + j * 32, H);
  }
}

// ---------------------------------------------------------------------------
// helpers of the lane-pair kernel
// ---------------------------------------------------------------------------

// Block count and boundary block of a request, used to keep the waves of a
// workgroup in lockstep: every wave decides trip counts and boundary
// iterations over all requests of the workgroup.
struct ReqPeek {
  int64_t nf;
  int64_t kr;  // iteration of the boundary block, else -1
};

template <int MODE>
__device__ __forceinline__ ReqPeek req_peek(const ChainArgs &a, int32_t i) {
  ReqPeek p{0, -1};
  if (i < a.n) {
    ChainReq q;
    const int32_t r = a.order ? a.order[i] : i;
    if (chain_setup<MODE>(a, r, q)) p = ReqPeek{q.nf, q.kr};
  }
  return p;
}

// ---------------------------------------------------------------------------
// lane-pair chain kernel
// ---------------------------------------------------------------------------
//
// A chain is latency-bound: the 64 rounds of a compression are a dependency
// chain, and with one lane per request a round costs its wave 14
// instructions (plus 10 per schedule word).  This kernel takes the message
// schedule off the rounds lanes and splits each round over two lanes.
// Write A_t for the word a after round t and E_t for e (so b_t = A_{t-1},
// c_t = A_{t-2}, d_t = A_{t-3}, and likewise f, g, h from E).  A round is
//   E_{t+1} = A_{t-3} + T1_t,   T1_t = E_{t-3} + Sigma1(E_t) + Ch(E_t, E_{t-1}, E_{t-2}) + K_t + W_t
//   A_{t+1} = T1_t + Sigma0(A_t) + Maj(A_t, A_{t-1}, A_{t-2})
//           = E_{t+1} - A_{t-3} + Sigma0(A_t) + Maj(A_t, A_{t-1}, A_{t-2}).
// Each request has two adjacent lanes of a rounds wave: the E lane (even)
// produces the E words and the A lane (odd) the A words, two rounds behind:
// in step i the E lane computes E_{i+1} and the A lane A_{i-1}.  Both run the
// same nine instructions on their own last four words x0..x3 (E: E_i..E_{i-3};
// A: A_{i-2}..A_{i-5}), and each needs its partner's x1 (A_{i-3} resp.
// E_{i-1}), which one DPP quad swap delivers to both:
//   S  = rotr(x0,r1) ^ rotr(x0,r2) ^ rotr(x0,r3)   Sigma1(E_i)          | Sigma0(A_{i-2})
//   X  = bitop(x0, x1, m)                          E_i                  | ~(A_{i-2} ^ A_{i-3})
//   F  = choose(X, x1, x2)                         Ch(E_i, .., ..)      | Maj(A_{i-2}, .., ..)
//   Z  = (x3 ^ m) + kw + partner's x1              E_{i-3} + K_i + W_i  | ~A_{i-5} + 1 + E_{i-1}
//                                                  + A_{i-3}            |
//   x0 = S + F + Z                                 E_{i+1}              | A_{i-1}
// with per-lane rotation amounts, m = 0 (E) or ~0 (A), and kw = K + W on E
// lanes and 1 on A lanes (a constant column of the LDS tables).  Choose with
// ~(a ^ b) as selector is Maj(a, b, c).  Z depends only on words from
// earlier steps, so it is formed one step ahead, and the DPP read is off the
// dependency chain (x0 -> rotates -> xor3 -> add3, and x0 -> X -> choose).
// A compression takes 66 steps: in steps 0 and 1 the A lane has nothing to
// compute (its x0 is then set to the initial b, then a; it starts from c, d),
// and in steps 64 and 65 only the A lane computes (A_63, A_64).
//
// Workgroup: 64 requests.  Waves 0 and 1 run the rounds of 32 requests each;
// wave 2 ("schedule", one lane per request) writes K + W of both
// compressions to LDS tables [round][request].  Per block j, C1 = (IV;
// h_{j-1} || T[0..7]) and C2 = (state; T[8..15] || padding):
//   phase 1  rounds: C1 rounds 0-11      schedule: reads h_{j-1}, C1's W[16..31]
//   phase 2  rounds: C1 rounds 12-27     schedule: C1's W[32..47]
//   phase 3  rounds: C1 rounds 28-43     schedule: C1's W[48..63]
//   phase 4  rounds: C1 rounds 44-63 and all of C2, then h_j to LDS and the
//            digest; schedule: the words of block j+1 that depend on tokens
//            only (C1 rounds 8-15, all of C2), double buffered by parity
// with a workgroup barrier after each phase; each barrier sits four rounds
// before the words it releases are needed, so that their LDS reads overlap
// those rounds.  The first compression's K + W of rounds 0..7 (the words of
// h_{j-1}) are formed by the rounds lanes from the LDS copy of h_{j-1},
// whose constant column holds 1 - K[t], so that the A lanes' sum is 1 there
// as well.  Iterations where some request of the workgroup has a special
// block run on the E lanes alone (rolled compressions) while the schedule
// wave prepares the next block.  All three waves derive trip counts and
// special iterations from all 64 requests, so they meet the same barriers.

constexpr int kLpCols = kWave + 1;  // 64 requests + the constant column
constexpr int kLpThreads = 3 * kWave;

struct LpLds {
  uint32_t ha[8][kLpCols];      // message words 0..7 of the first compression;
                                // constant column: 1 - K[t]
  uint32_t hb[8][kLpCols];      // message words 8..15; constant column: 1 - K[8 + t]
  uint32_t c1b[48][kLpCols];    // K + W of the first compression, rounds 16..63
  uint32_t c2[2][64][kLpCols];  // K + W of the second compression, by block parity
  uint32_t c3[64][2];           // K + W of a 128-byte message's padding block; [.][1] = 1
};
constexpr int kLpRows = 8 + 8 + 48 + 128;  // rows with a constant column
static_assert(sizeof(LpLds) == (size_t)kLpRows * kLpCols * 4 + 64 * 2 * 4,
              "LpLds rows are contiguous");

// K + W of the padding block of a 128-byte message (constant), from the
// schedule's definition
struct PadSchedule {
  uint32_t kw[64];
};
constexpr uint32_t c_rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }
constexpr PadSchedule make_pad128_schedule() {
  PadSchedule p{};
  uint32_t w[64] = {};
  w[0] = 0x80000000u;
  w[15] = 128 * 8;
  for (int t = 16; t < 64; ++t) {
    const uint32_t s0 = c_rotr(w[t - 15], 7) ^ c_rotr(w[t - 15], 18) ^ (w[t - 15] >> 3);
    const uint32_t s1 = c_rotr(w[t - 2], 17) ^ c_rotr(w[t - 2], 19) ^ (w[t - 2] >> 10);
    w[t] = s1 + w[t - 7] + s0 + w[t - 16];
  }
  for (int t = 0; t < 64; ++t) p.kw[t] = kSha.K[t] + w[t];
  return p;
}
__constant__ PadSchedule kPad128Dev = make_pad128_schedule();

struct LpLane {
  uint32_t r1, r2, r3;  // rotation amounts of the lane's big sigma
  uint32_t m;           // 0 on E lanes, ~0 on A lanes
};

// the partner lane's x (adjacent lanes swap: DPP quad_perm [1,0,3,2])
__device__ __forceinline__ uint32_t lp_partner(uint32_t x) {
  return __builtin_amdgcn_update_dpp(0u, x, 0xB1, 0xF, 0xF, false);
}

// z of a compression's step 0: (x3 ^ m) + kw_0 + the partner's x1
__device__ __forceinline__ uint32_t lp_z0(const uint32_t s[4], uint32_t kw0, const LpLane &c) {
  uint32_t z = (s[3] ^ c.m) + kw0;
  asm("" : "+v"(z));  // keeps the partner term one DPP add
  return z + lp_partner(s[1]);
}

// One step, or two in one block.  On entry z holds this step's Z; a step
// forms x0' and the next step's Z from kwn (the next step's x3 is this
// step's x2, and its partner's x1 is the partner's present x0).  Written as
// asm so that no instruction waits on the one before it, except the first
// on the previous step's x0.  The DPP source (x0) was written at least one
// step earlier (nine instructions), so the DPP read needs no wait states.
#define KVGOV_LP_STEP(X0, X1, X2, Z, V, ZN, KWN, T1, T2, T3, XX, F, S)               \
  "v_alignbit_b32 " T1 ", " X0 ", " X0 ", %[r1]\n\t"                              \
  "v_alignbit_b32 " T2 ", " X0 ", " X0 ", %[r2]\n\t"                              \
  "v_bitop3_b32 " XX ", " X0 ", " X1 ", %[m] bitop3:0xd2\n\t"                     \
  "v_alignbit_b32 " T3 ", " X0 ", " X0 ", %[r3]\n\t"                              \
  "v_bitop3_b32 " F ", " XX ", " X1 ", " X2 " bitop3:0xca\n\t"                    \
  "v_bitop3_b32 " S ", " T1 ", " T2 ", " T3 " bitop3:0x96\n\t"                    \
  "v_xad_u32 " ZN ", " X2 ", %[m], " KWN "\n\t"                                   \
  "v_add3_u32 " V ", " S ", " F ", " Z "\n\t"                                     \
  "v_add_u32_dpp " ZN ", " X0 ", " ZN " quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"

__device__ __forceinline__ void lp_step(uint32_t s[4], uint32_t &z, uint32_t kwn,
                                        const LpLane &c) {
  uint32_t t1, t2, t3, x, f, sg, v, zn;
  asm(KVGOV_LP_STEP("%[x0]", "%[x1]", "%[x2]", "%[z]", "%[v]", "%[zn]", "%[kwn]", "%[t1]",
                    "%[t2]", "%[t3]", "%[x]", "%[f]", "%[sg]")
      : [t1] "=&v"(t1), [t2] "=&v"(t2), [x] "=&v"(x), [t3] "=&v"(t3), [f] "=&v"(f),
        [sg] "=&v"(sg), [zn] "=&v"(zn), [v] "=&v"(v)
      : [x0] "v"(s[0]), [x1] "v"(s[1]), [x2] "v"(s[2]), [z] "v"(z), [m] "v"(c.m),
        [r1] "v"(c.r1), [r2] "v"(c.r2), [r3] "v"(c.r3), [kwn] "v"(kwn));
  s[3] = s[2];
  s[2] = s[1];
  s[1] = s[0];
  s[0] = v;
  z = zn;
}

__device__ __forceinline__ void lp_step2(uint32_t s[4], uint32_t &z, uint32_t kwn1,
                                         uint32_t kwn2, const LpLane &c) {
  uint32_t t1, t2, t3, x, f, sg, u1, u2, u3, y, g, sh, va, vb, za, zb;
  asm(KVGOV_LP_STEP("%[x0]", "%[x1]", "%[x2]", "%[z]", "%[va]", "%[za]", "%[k1]", "%[t1]",
                    "%[t2]", "%[t3]", "%[x]", "%[f]", "%[sg]")
      KVGOV_LP_STEP("%[va]", "%[x0]", "%[x1]", "%[za]", "%[vb]", "%[zb]", "%[k2]", "%[u1]",
                    "%[u2]", "%[u3]", "%[y]", "%[g]", "%[sh]")
      : [t1] "=&v"(t1), [t2] "=&v"(t2), [x] "=&v"(x), [t3] "=&v"(t3), [f] "=&v"(f),
        [sg] "=&v"(sg), [za] "=&v"(za), [va] "=&v"(va), [u1] "=&v"(u1), [u2] "=&v"(u2),
        [y] "=&v"(y), [u3] "=&v"(u3), [g] "=&v"(g), [sh] "=&v"(sh), [zb] "=&v"(zb),
        [vb] "=&v"(vb)
      : [x0] "v"(s[0]), [x1] "v"(s[1]), [x2] "v"(s[2]), [z] "v"(z), [m] "v"(c.m),
        [r1] "v"(c.r1), [r2] "v"(c.r2), [r3] "v"(c.r3), [k1] "v"(kwn1), [k2] "v"(kwn2));
  s[3] = s[1];
  s[2] = s[0];
  s[1] = va;
  s[0] = vb;
  z = zb;
}

// Runs of 6, 14 or 16 steps as one asm statement: the compiler puts a wait
// state between consecutive asm statements (it cannot see that their DPP
// sources are old), which cost about a cycle per step with two-step
// statements.  The four words x0..x3 live in a ring of four registers q0..q3
// (step k reads x0 from q[-k mod 4] and writes x0' over the dead x3), Z
// alternates between y0 and y1, and six temporaries are reused by every
// step.  After a multiple of four steps the ring is back in place; after
// 4k + 2 steps x0..x3 sit in q2, q3, q0, q1.
#define KVGOV_LP_RING_T "%[t1]", "%[t2]", "%[t3]", "%[x]", "%[f]", "%[sg]"
#define KVGOV_LP_STEP_(...) KVGOV_LP_STEP(__VA_ARGS__)
#define KVGOV_LP_R0(K) KVGOV_LP_STEP_("%[q0]", "%[q1]", "%[q2]", "%[y0]", "%[q3]", "%[y1]", K, KVGOV_LP_RING_T)
#define KVGOV_LP_R1(K) KVGOV_LP_STEP_("%[q3]", "%[q0]", "%[q1]", "%[y1]", "%[q2]", "%[y0]", K, KVGOV_LP_RING_T)
#define KVGOV_LP_R2(K) KVGOV_LP_STEP_("%[q2]", "%[q3]", "%[q0]", "%[y0]", "%[q1]", "%[y1]", K, KVGOV_LP_RING_T)
#define KVGOV_LP_R3(K) KVGOV_LP_STEP_("%[q1]", "%[q2]", "%[q3]", "%[y1]", "%[q0]", "%[y0]", K, KVGOV_LP_RING_T)
#define KVGOV_LP_RING4(A, B, C, D) KVGOV_LP_R0(A) KVGOV_LP_R1(B) KVGOV_LP_R2(C) KVGOV_LP_R3(D)
#define KVGOV_LP_RING_OUT                                                                    \
  [q0] "+v"(s[0]), [q1] "+v"(s[1]), [q2] "+v"(s[2]), [q3] "+v"(s[3]), [y0] "+v"(z),         \
      [y1] "=&v"(y1), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3), [x] "=&v"(x),          \
      [f] "=&v"(f), [sg] "=&v"(sg)
#define KVGOV_LP_RING_IN [m] "v"(c.m), [r1] "v"(c.r1), [r2] "v"(c.r2), [r3] "v"(c.r3)
#define KVGOV_LP_K(i) [k##i] "v"(k[i - 1])

// k[i] is the kw taken by step i (the next step's)
template <int N>
__device__ __forceinline__ void lp_ring(uint32_t s[4], uint32_t &z, const uint32_t k[N],
                                        const LpLane &c) {
  static_assert(N == 6 || N == 14 || N == 16, "ring runs of 6, 14 or 16 steps");
  uint32_t y1, t1, t2, t3, x, f, sg;
  if constexpr (N == 16) {
    asm(KVGOV_LP_RING4("%[k1]", "%[k2]", "%[k3]", "%[k4]")
        KVGOV_LP_RING4("%[k5]", "%[k6]", "%[k7]", "%[k8]")
        KVGOV_LP_RING4("%[k9]", "%[k10]", "%[k11]", "%[k12]")
        KVGOV_LP_RING4("%[k13]", "%[k14]", "%[k15]", "%[k16]")
        : KVGOV_LP_RING_OUT
        : KVGOV_LP_RING_IN, KVGOV_LP_K(1), KVGOV_LP_K(2), KVGOV_LP_K(3), KVGOV_LP_K(4),
          KVGOV_LP_K(5), KVGOV_LP_K(6), KVGOV_LP_K(7), KVGOV_LP_K(8), KVGOV_LP_K(9),
          KVGOV_LP_K(10), KVGOV_LP_K(11), KVGOV_LP_K(12), KVGOV_LP_K(13), KVGOV_LP_K(14),
          KVGOV_LP_K(15), KVGOV_LP_K(16));
  } else if constexpr (N == 14) {
    asm(KVGOV_LP_RING4("%[k1]", "%[k2]", "%[k3]", "%[k4]")
        KVGOV_LP_RING4("%[k5]", "%[k6]", "%[k7]", "%[k8]")
        KVGOV_LP_RING4("%[k9]", "%[k10]", "%[k11]", "%[k12]")
        KVGOV_LP_R0("%[k13]") KVGOV_LP_R1("%[k14]")
        : KVGOV_LP_RING_OUT
        : KVGOV_LP_RING_IN, KVGOV_LP_K(1), KVGOV_LP_K(2), KVGOV_LP_K(3), KVGOV_LP_K(4),
          KVGOV_LP_K(5), KVGOV_LP_K(6), KVGOV_LP_K(7), KVGOV_LP_K(8), KVGOV_LP_K(9),
          KVGOV_LP_K(10), KVGOV_LP_K(11), KVGOV_LP_K(12), KVGOV_LP_K(13), KVGOV_LP_K(14));
  } else {
    asm(KVGOV_LP_RING4("%[k1]", "%[k2]", "%[k3]", "%[k4]")
        KVGOV_LP_R0("%[k5]") KVGOV_LP_R1("%[k6]")
        : KVGOV_LP_RING_OUT
        : KVGOV_LP_RING_IN, KVGOV_LP_K(1), KVGOV_LP_K(2), KVGOV_LP_K(3), KVGOV_LP_K(4),
          KVGOV_LP_K(5), KVGOV_LP_K(6));
  }
  if constexpr (N % 4 == 2) {
    const uint32_t w0 = s[2], w1 = s[3], w2 = s[0], w3 = s[1];
    s[0] = w0;
    s[1] = w1;
    s[2] = w2;
    s[3] = w3;
  }
}

// N steps; kw holds the group's own kw (kw[0] is already in z), kw_after
// the kw of the step after the group
template <int N>
__device__ __forceinline__ void lp_steps(uint32_t s[4], uint32_t &z, const uint32_t *kw,
                                         uint32_t kw_after, const LpLane &c) {
  if constexpr (N == 6 || N == 14 || N == 16) {
    uint32_t k[N];
#pragma unroll
    for (int i = 0; i < N; ++i) k[i] = i + 1 < N ? kw[i + 1] : kw_after;
    lp_ring<N>(s, z, k, c);
  } else {
#pragma unroll
    for (int i = 0; i + 1 < N; i += 2)
      lp_step2(s, z, kw[i + 1], i + 2 < N ? kw[i + 2] : kw_after, c);
    if (N & 1) lp_step(s, z, kw_after, c);
  }
}

// steps 0 and 1 of a compression: the A lane's results are replaced by the
// initial b, then a
__device__ __forceinline__ void lp_head(uint32_t s[4], uint32_t &z, uint32_t kw1, uint32_t kw2,
                                        const LpLane &c, uint32_t b0, uint32_t a0,
                                        bool a_lane) {
  lp_step(s, z, kw1, c);
  s[0] = a_lane ? b0 : s[0];
  lp_step(s, z, kw2, c);
  s[0] = a_lane ? a0 : s[0];
}

// steps 64 and 65: the A lane computes A_63 and A_64; the E lane's words
// were final after step 63 (e..h), the A lane's after step 65 (a..d)
__device__ __forceinline__ void lp_tail(uint32_t s[4], uint32_t &z, const LpLane &c,
                                        bool a_lane) {
  uint32_t e[4];
#pragma unroll
  for (int x = 0; x < 4; ++x) e[x] = s[x];
  lp_step2(s, z, 1u, 1u, c);
#pragma unroll
  for (int x = 0; x < 4; ++x) s[x] = a_lane ? s[x] : e[x];
}

__device__ __forceinline__ void lp_load16(uint32_t w[16], const uint32_t (*rows)[kLpCols],
                                          int base, int col) {
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = rows[base + i][col];
}

// schedule words W[t0..t0+15] from the rolling window w (W[t0-16..t0-1]);
// stores K[t0 + i] + W[t0 + i] to rows[base + i][lane]
template <int T0>
__device__ __forceinline__ void lp_sched16(uint32_t w[16], uint32_t (*rows)[kLpCols], int base,
                                           int lane) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    w[i] = small_sigma1(w[(i + 14) & 15]) + w[(i + 9) & 15] + small_sigma0(w[(i + 1) & 15]) +
           w[i];
    rows[base + i][lane] = w[i] + kSha.K[T0 + i];
  }
}

// schedule words W[T0..T0+N-1] (T0 >= 16) from the rolling window w, which
// holds W[t] at w[t & 15]; stores K[t] + W[t] to rows[t - 16][lane].  With
// PRE, the terms of W[16..30] that depend on message words 8..15 alone come
// from pre (lp_presum), computed while the previous block was hashed.
template <int T0, int N, bool PRE>
__device__ __forceinline__ void lp_sched_words(uint32_t w[16], uint32_t (*rows)[kLpCols],
                                               int lane, const uint32_t pre[16]) {
#pragma unroll
  for (int t = T0; t < T0 + N; ++t) {
    uint32_t v;
    if (PRE && (t == 16 || t == 17))
      v = small_sigma0(w[(t - 15) & 15]) + w[t & 15] + pre[t - 16];
    else if (PRE && t == 23)
      v = small_sigma1(w[(t - 2) & 15]) + w[(t - 7) & 15] + pre[7] + w[t & 15];
    else if (PRE && t >= 24 && t <= 30)
      v = small_sigma1(w[(t - 2) & 15]) + w[(t - 7) & 15] + pre[t - 16];
    else
      v = small_sigma1(w[(t - 2) & 15]) + w[(t - 7) & 15] + small_sigma0(w[(t - 15) & 15]) +
          w[t & 15];
    w[t & 15] = v;
    rows[t - 16][lane] = v + kSha.K[t];
  }
}

// The parts of schedule words 16..30 of a first compression whose message
// words 8..15 are m[0..7] (every block but the chain's first and the
// boundary block) that do not involve words 0..7:
//   W16 = sigma0(W1) + W0 + [sigma1(W14) + W9]     W17 likewise
//   W23 = sigma1(W21) + W16 + W7 + [sigma0(W8)]
//   W24..W30 = sigma1(W[t-2]) + W[t-7] + [sigma0(W[t-15]) + W[t-16]]
__device__ __forceinline__ void lp_presum(const uint32_t m[8], uint32_t pre[16]) {
  pre[0] = small_sigma1(m[6]) + m[1];
  pre[1] = small_sigma1(m[7]) + m[2];
  pre[7] = small_sigma0(m[0]);
#pragma unroll
  for (int i = 0; i < 7; ++i) pre[8 + i] = small_sigma0(m[1 + i]) + m[i];
}

// The first compression's schedule words W[16..63] depend on h_{j-1} and are
// released to the rounds waves in groups, one barrier each: group g holds
// W[kLpGroup[g] .. kLpGroup[g + 1] - 1].  A barrier costs the waves about as
// much as the rounds lose waiting for a larger group (the schedule wave
// makes a word a little slower than the rounds use one): three groups of 16
// measured fastest, splits into 4 to 8 groups slower.
constexpr int kLpGroup[] = {KVGOV_LP_GROUPS};
constexpr int kLpGroups = (int)(sizeof(kLpGroup) / sizeof(kLpGroup[0])) - 1;
static_assert(kLpGroup[0] == 16 && kLpGroup[kLpGroups] == 64, "groups cover W[16..63]");

template <int G>
__device__ __forceinline__ void lp_sched_groups(uint32_t w[16], uint32_t (*rows)[kLpCols],
                                                int lane, bool work, const uint32_t pre[16],
                                                bool use_pre) {
  if constexpr (G < kLpGroups) {
    constexpr int S = kLpGroup[G], N = kLpGroup[G + 1] - kLpGroup[G];
    static_assert(N > 0, "groups ascend");
    if (work) {
      if (S <= 30 && use_pre)  // workgroup-uniform
        lp_sched_words<S, N, true>(w, rows, lane, pre);
      else
        lp_sched_words<S, N, false>(w, rows, lane, pre);
    }
    __syncthreads();
    lp_sched_groups<G + 1>(w, rows, lane, work, pre, use_pre);
  }
}

// Rounds of the first compression from step kLpGroup[G] - C on: after the
// barrier that releases group G, its K + W rows are loaded into kw and the
// steps up to the next group's barrier (or to step 63) run.  kw2 receives
// the second compression's first 16 K + W rows during the last group.
template <int G>
__device__ __forceinline__ void lp_round_groups(uint32_t s[4], uint32_t &z, uint32_t kw[64],
                                                uint32_t kw2[16],
                                                const uint32_t (*rows)[kLpCols],
                                                const uint32_t (*rows2)[kLpCols], int col,
                                                const LpLane &c, bool act) {
  if constexpr (G < kLpGroups) {
    constexpr int C = KVGOV_LP_COVER;
    constexpr int S = kLpGroup[G], E = kLpGroup[G + 1];
    __syncthreads();  // releases W[S..E-1]
    if (act) {
#pragma unroll
      for (int t = S; t < E; ++t) kw[t] = rows[t - 16][col];
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (E < 64) {
        lp_steps<E - S>(s, z, kw + S - C, kw[E - C], c);
      } else {
        lp_steps<C>(s, z, kw + S - C, kw[S], c);
        lp_load16(kw2, rows2, 0, col);
        __builtin_amdgcn_sched_barrier(0);
        lp_steps<64 - S>(s, z, kw + S, 1u, c);
      }
    }
    lp_round_groups<G + 1>(s, z, kw, kw2, rows, rows2, col, c, act);
  }
}

// Message schedule on a lane pair: with two schedule lanes per request,
// lane p of the pair makes the words W[t], t = 16 + 2k + p, of step k, so a
// wave makes a word of 32 requests in about 16 instructions per two words
// instead of one lane making every word in 11.  Both lanes keep a 16-word
// window in which lane p's logical word i at step k is W[2k + p + i],
// stored at w[(2k + i) & 15]: the four operands of W[t] (t - 16, t - 15,
// t - 7, t - 2: logical 0, 1, 9, 14) are then the same registers on both
// lanes.  After the step each lane takes its partner's new word with one DPP
// swap: lane 0 needs it as logical 15 of the next window (W[17 + 2k]), lane 1
// as logical 13 (W[16 + 2k]); lane 1's logical 15 (W[18 + 2k], lane 0's next
// word) is set the same way one step later, before it is first read (as
// logical 9, four steps on).  rows[2k + p][col] receives K[t] + W[t].
template <int K>
__device__ __forceinline__ void lp_pair_step(uint32_t w[16], uint32_t (*rows)[kLpCols], int col,
                                             bool odd) {
  constexpr int i0 = (2 * K) & 15, i1 = (2 * K + 1) & 15, i9 = (2 * K + 9) & 15;
  constexpr int i14 = (2 * K + 14) & 15, i15 = (2 * K + 15) & 15;
  const uint32_t v = small_sigma1(w[i14]) + w[i9] + small_sigma0(w[i1]) + w[i0];
  const uint32_t kt = odd ? kSha.K[17 + 2 * K] : kSha.K[16 + 2 * K];
  rows[2 * K + (odd ? 1 : 0)][col] = v + kt;
  const uint32_t pv = lp_partner(v);
  w[i0] = v;                    // logical 14 of the next window
  w[i1] = pv;                   // logical 15 (lane 1: replaced before it is read)
  w[i15] = odd ? pv : w[i15];   // logical 13 on lane 1
}

// Steps K .. K + N - 1.
template <int K, int N>
__device__ __forceinline__ void lp_pair_run(uint32_t w[16], uint32_t (*rows)[kLpCols], int col,
                                            bool odd) {
  if constexpr (N > 0) {
    lp_pair_step<K>(w, rows, col, odd);
    lp_pair_run<K + 1, N - 1>(w, rows, col, odd);
  }
}

// The window of step 0 from the message words m[0..15] (all on both lanes):
// lane 1's logical i is W[i + 1]; its logical 15 (W[16]) comes from lane 0's
// first step.
__device__ __forceinline__ void lp_pair_window(const uint32_t m[16], uint32_t w[16], bool odd) {
#pragma unroll
  for (int i = 0; i < 15; ++i) w[i] = odd ? m[i + 1] : m[i];
  w[15] = m[15];
}

// The first compression's schedule in groups, as lp_sched_groups, on lane
// pairs: group g's words, then the barrier that releases them.
template <int G>
__device__ __forceinline__ void lp_pair_groups(uint32_t w[16], uint32_t (*rows)[kLpCols], int col,
                                               bool odd, bool work) {
  if constexpr (G < kLpGroups) {
    constexpr int S = kLpGroup[G], N = kLpGroup[G + 1] - kLpGroup[G];
    static_assert(S % 2 == 0 && N % 2 == 0, "pair groups hold whole steps");
    if (work) lp_pair_run<(S - 16) / 2, N / 2>(w, rows, col, odd);
    __syncthreads();
    lp_pair_groups<G + 1>(w, rows, col, odd, work);
  }
}

// Per block and request, the three message patterns of the chain (the
// compressions of a block, "first" and "second", plus a third for the
// boundary block):
//   plain        first (IV; h_{j-1} || T[0..7])   second (.; T[8..15] || pad96)
//   first block  first (IV; T[0..15])             second (.; pad64)
//   boundary     first (IV; sigma || h_{k-1})     second (.; T[0..15])
//                third (.; pad128)
// Prepared one block ahead from tokens and constants: the first message's
// words into ha / hb except h_{j-1} (written by the rounds lanes at the end
// of block j - 1), and K + W of all 64 rounds of the second message.
__device__ __forceinline__ void lp_message(const uint32_t Tn[16], const uint32_t sig[8],
                                           bool first_block, bool boundary, LpLds &L, int buf,
                                           int lane, uint32_t m[16]) {
  if (boundary) {
#pragma unroll
    for (int x = 0; x < 8; ++x) L.ha[x][lane] = sig[x];
#pragma unroll
    for (int x = 0; x < 16; ++x) m[x] = Tn[x];
  } else if (first_block) {
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      L.ha[x][lane] = Tn[x];
      L.hb[x][lane] = Tn[8 + x];
    }
    m[0] = 0x80000000u;
#pragma unroll
    for (int x = 1; x < 15; ++x) m[x] = 0;
    m[15] = 64 * 8;
  } else {
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      L.hb[x][lane] = Tn[x];
      m[x] = Tn[8 + x];
    }
    pad96_tail(m);
  }
#pragma unroll
  for (int x = 0; x < 16; ++x) L.c2[buf][x][lane] = kSha.K[x] + m[x];
}

__device__ __forceinline__ void lp_prepare(const uint32_t Tn[16], const uint32_t sig[8],
                                           bool first_block, bool boundary, LpLds &L, int buf,
                                           int lane) {
  uint32_t m[16];
  lp_message(Tn, sig, first_block, boundary, L, buf, lane, m);
  lp_sched16<16>(m, L.c2[buf], 16, lane);
  lp_sched16<32>(m, L.c2[buf], 32, lane);
  lp_sched16<48>(m, L.c2[buf], 48, lane);
}

// lp_prepare on a lane pair: both lanes write the same message words (the
// same values to the same addresses), the schedule is split by parity.
__device__ __forceinline__ void lp_prepare_pair(const uint32_t Tn[16], const uint32_t sig[8],
                                                bool first_block, bool boundary, LpLds &L, int buf,
                                                int col, bool odd) {
  uint32_t m[16], w[16];
  lp_message(Tn, sig, first_block, boundary, L, buf, col, m);
  lp_pair_window(m, w, odd);
  lp_pair_run<0, 24>(w, L.c2[buf] + 16, col, odd);
}

__device__ __forceinline__ void lp_load16(uint32_t w[16], const uint32_t (*rows)[2], int base,
                                          int col) {
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i] = rows[base + i][col];
}

// The rounds of one compression from the initial words st (E: e..h, A:
// a..d), K + W from 16-row groups: kw0 holds rounds 0..15 (already in
// registers), the later groups are loaded from `rows` (64 rows) one group
// ahead; returns st + the compression's result.
template <typename Rows>
__device__ __forceinline__ void lp_compress_rows(uint32_t st[4], const uint32_t kw0[16], Rows rows,
                                                 int col, const LpLane &c, bool a_lane) {
  uint32_t s[4], wa[16], wb[16], z;
#pragma unroll
  for (int x = 0; x < 4; ++x) s[x] = a_lane ? (x < 2 ? st[x + 2] : 0u) : st[x];
  z = lp_z0(s, kw0[0], c);
  lp_load16(wa, rows, 16, col);
  __builtin_amdgcn_sched_barrier(0);
  lp_head(s, z, kw0[1], kw0[2], c, st[1], st[0], a_lane);
  lp_steps<14>(s, z, kw0 + 2, wa[0], c);   // 2..15
  lp_load16(wb, rows, 32, col);
  __builtin_amdgcn_sched_barrier(0);
  lp_steps<16>(s, z, wa, wb[0], c);        // 16..31
  lp_load16(wa, rows, 48, col);
  __builtin_amdgcn_sched_barrier(0);
  lp_steps<16>(s, z, wb, wa[0], c);        // 32..47
  lp_steps<16>(s, z, wa, 1u, c);           // 48..63
  lp_tail(s, z, c, a_lane);
#pragma unroll
  for (int x = 0; x < 4; ++x) st[x] += s[x];
}

// Workgroup `group` of the lane-pair kernel: requests group * 64 + 0..63 of
// the (ordered) batch.  Waves 0 and 1 run the rounds.  PAIR (workgroups of
// four waves): waves 2 and 3 run the schedule with two lanes per request
// (32 requests each), so that the first compression's words are ready before
// the rounds take them; otherwise wave 2 runs it with one lane per request
// (and a fourth wave, if any, only keeps the barriers).
template <int MODE, bool PAIR>
__device__ __forceinline__ void lp_group(const ChainArgs &a, int32_t group, LpLds &L) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const bool sched_wave = wave >= 2;
  const bool idle = !PAIR && wave >= 3;
  const bool a_lane = !sched_wave && (lane & 1);
  // the lane's parity in a schedule pair
  const bool odd = PAIR && sched_wave && (lane & 1);
  // the request (LDS column) of this lane within the workgroup
  const int mine = sched_wave && !PAIR ? lane : (wave & 1) * 32 + (lane >> 1);
  const int32_t base = group * kWave;
  const int32_t i = base + mine;

  ChainReq q;
  bool ok = false;
  if (i < a.n) {
    const int32_t r = a.order ? a.order[i] : i;
    ok = chain_setup<MODE>(a, r, q);
  }
  const int64_t nf = ok ? q.nf : 0;
  const int64_t kb = ok ? q.kr : -1;  // boundary iteration (boundary mode), else -1
  // Trip count and boundary iterations are decided over all 64 requests of
  // the workgroup: the schedule wave holds them all, and a rounds lane also
  // looks at the request of the same lane in the other rounds wave.
  const ReqPeek own{nf, kb};
  ReqPeek other{0, -1};
  if (!sched_wave || PAIR) other = req_peek<MODE>(a, base + (1 - (wave & 1)) * 32 + (mine & 31));
  int64_t J = own.nf > other.nf ? own.nf : other.nf;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    const int64_t o = __shfl_xor(J, d, kWave);
    J = o > J ? o : J;
  }

  // constant columns; the padding block of a 128-byte message
  uint32_t(*rows)[kLpCols] = reinterpret_cast<uint32_t(*)[kLpCols]>(&L);
  for (int x = threadIdx.x; x < kLpRows; x += blockDim.x)
    rows[x][kWave] = x < 16 ? 1u - kShaDev.K[x] : 1u;
  for (int x = threadIdx.x; x < 64; x += blockDim.x) {
    L.c3[x][0] = kPad128Dev.kw[x];
    L.c3[x][1] = 1u;
  }

  // rounds lanes: role constants
  LpLane c;
  c.r1 = a_lane ? 2 : 6;
  c.r2 = a_lane ? 13 : 11;
  c.r3 = a_lane ? 22 : 25;
  c.m = a_lane ? ~0u : 0u;
  const int col = a_lane ? kWave : mine;
  const int col3 = a_lane ? 1 : 0;
  const int half = a_lane ? 0 : 4;  // state words held: a..d = 0..3, e..h = 4..7
  uint32_t iv[4];                   // the initial value's words held by the lane
#pragma unroll
  for (int x = 0; x < 4; ++x) iv[x] = a_lane ? kSha.H0[x] : kSha.H0[4 + x];

  // schedule wave: tokens one block ahead (lanes without blocks read a
  // valid dummy block: the loop runs only if some request of the workgroup
  // has a block, so the token array holds at least 16 tokens)
  u32x4 nxt[4];
  const int32_t *tp = nf > 0 ? q.tp : a.tokens;
  const int64_t nfl = nf > 0 ? nf : 1;
  if (sched_wave && !idle && J > 0) {
    load_raw(tp, nxt);
    uint32_t T0[16];
    take_block(nxt, T0, tp, 0, nfl);
    if (nf > 0) {
      // h_{j0-1}: the parent digest when resuming (in the second half of a
      // boundary block's first message), sigma for a salted root
      const bool resume = q.j0 > 0, bnd0 = MODE == KVGOV_BOUNDARY && kb == 0;
      if (resume || q.salted_root) {
        uint32_t h[8];
        if (resume)
          load_digest(a.parents + (int64_t)(a.order ? a.order[i] : i) * 32, h);
#pragma unroll
        for (int x = 0; x < 8; ++x) (bnd0 ? L.hb : L.ha)[x][mine] = resume ? h[x] : q.sig[x];
      }
      if (PAIR)
        lp_prepare_pair(T0, q.sig, !resume && !q.salted_root, bnd0, L, 0, mine, odd);
      else
        lp_prepare(T0, q.sig, !resume && !q.salted_root, bnd0, L, 0, lane);
    }
  }
  __syncthreads();

  uint32_t pre[16];  // schedule lanes: partial sums of the next block's first schedule
#pragma unroll
  for (int x = 0; x < 16; ++x) pre[x] = 0;
  for (int64_t j = 0; j < J; ++j) {
    const bool act = j < nf;
    const bool next = j + 1 < nf;
    const int cb = (int)(j & 1), nb = cb ^ 1;
    // boundary blocks take a third compression (workgroup-uniform decision)
    bool third = false;
    if (MODE == KVGOV_BOUNDARY) {
      const bool mine_bnd = (j < own.nf && j == own.kr) || (j < other.nf && j == other.kr);
      third = __any(mine_bnd);
    }

    if (!sched_wave) {
      // ---- rounds waves.  Step i of a group takes the kw of step i + 1 (the
      // next step's z starts early).  Each barrier comes C steps before the
      // first word it releases is taken, so that the LDS reads after it are
      // covered by those steps.
      constexpr int C = KVGOV_LP_COVER;
      uint32_t s[4], st[4], wa[16], z = 0;
      uint32_t kw[64];
      if (act) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          kw[t] = kSha.K[t] + L.ha[t][col];
          kw[8 + t] = kSha.K[8 + t] + L.hb[t][col];
        }
#pragma unroll
        for (int x = 0; x < 4; ++x) s[x] = a_lane ? (x < 2 ? iv[x + 2] : 0u) : iv[x];
        z = lp_z0(s, kw[0], c);
        lp_head(s, z, kw[1], kw[2], c, iv[1], iv[0], a_lane);
        lp_steps<6>(s, z, kw + 2, kw[8], c);  // steps 2..7
        lp_steps<8 - C>(s, z, kw + 8, kw[16 - C], c);
      }
      // steps 16 - C .. 63, one barrier per schedule group
      lp_round_groups<0>(s, z, kw, wa, L.c1b, L.c2[cb], col, c, act);
      if (act) {
        lp_tail(s, z, c, a_lane);
#pragma unroll
        for (int x = 0; x < 4; ++x) st[x] = iv[x] + s[x];
        // second compression
        lp_compress_rows(st, wa, L.c2[cb], col, c, a_lane);
        if (MODE == KVGOV_BOUNDARY && third) {
          // third compression (the boundary block's padding), for all lanes;
          // only boundary requests keep its result
          uint32_t st3[4], k3[16];
#pragma unroll
          for (int x = 0; x < 4; ++x) st3[x] = st[x];
          lp_load16(k3, L.c3, 0, col3);
          lp_compress_rows(st3, k3, L.c3, col3, c, a_lane);
          const bool bnd = j == kb;
#pragma unroll
          for (int x = 0; x < 4; ++x) st[x] = bnd ? st3[x] : st[x];
        }
        // h_j: the next block's first message words 0..7 (plain), or 8..15
        // (the next block is the boundary block)
        const bool next_bnd = MODE == KVGOV_BOUNDARY && j + 1 == kb;
        uint32_t(*hrows)[kLpCols] = next_bnd ? L.hb : L.ha;
#pragma unroll
        for (int x = 0; x < 4; ++x) hrows[half + x][mine] = st[x];
        u32x4 *dst = reinterpret_cast<u32x4 *>(q.out + j * 32 + half * 4);
        *dst = u32x4{bswap(st[0]), bswap(st[1]), bswap(st[2]), bswap(st[3])};
      }
      __syncthreads();
    } else if (PAIR) {
      // ---- schedule waves, two lanes per request
      uint32_t w[16];
      if (act) {
        uint32_t m[16];
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          m[x] = L.ha[x][mine];
          m[8 + x] = L.hb[x][mine];
        }
        lp_pair_window(m, w, odd);
      }
      lp_pair_groups<0>(w, L.c1b, mine, odd, act);
      {
        // block j + 1's tokens, and the load of block j + 2
        uint32_t Tn[16];
        const int64_t jn = j + 1 < nfl ? j + 1 : nfl - 1;
        take_block(nxt, Tn, tp, jn, nfl);
        if (next) {
          const bool bnd_next = MODE == KVGOV_BOUNDARY && j + 1 == kb;
          lp_prepare_pair(Tn, q.sig, false, bnd_next, L, nb, mine, odd);
        }
      }
      __syncthreads();
    } else {
      // ---- schedule wave (an idle wave only meets the barriers)
      uint32_t w[16];
      if (act && !idle) {
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          w[x] = L.ha[x][lane];
          w[8 + x] = L.hb[x][lane];
        }
      }
      // the partial sums hold for block j unless it is a chain's first
      // block or some request's boundary block
      lp_sched_groups<0>(w, L.c1b, lane, act && !idle, pre, j > 0 && !third);
      if (!idle) {
        // block j + 1's tokens, and the load of block j + 2
        uint32_t Tn[16];
        const int64_t jn = j + 1 < nfl ? j + 1 : nfl - 1;
        take_block(nxt, Tn, tp, jn, nfl);
        if (next) {
          const bool bnd_next = MODE == KVGOV_BOUNDARY && j + 1 == kb;
          lp_prepare(Tn, q.sig, false, bnd_next, L, nb, lane);
          lp_presum(Tn, pre);
        }
      }
      __syncthreads();
    }
  }
}

template <int MODE, bool PAIR>
__global__ __launch_bounds__(4 * kWave) void k_chains_lp(ChainArgs a) {
  __shared__ LpLds L;
  lp_group<MODE, PAIR>(a, blockIdx.x, L);
}

// Large ordered batches: the first `lp_groups` workgroups run the lane-pair
// path on the longest requests (the batch is ordered longest first), so
// that the longest chains finish ~1.4x sooner; the remaining workgroups run
// one lane per request on the rest.  Both in one launch, 256 lanes per
// workgroup.
template <int MODE>
__global__ __launch_bounds__(256) void k_chains_mixed(ChainArgs a, int32_t lp_groups) {
  __shared__ LpLds L;
  if ((int32_t)blockIdx.x < lp_groups)
    lp_group<MODE, true>(a, blockIdx.x, L);
  else
    single_chain<MODE>(a, lp_groups * kWave + ((int32_t)blockIdx.x - lp_groups) * 256 +
                              (int32_t)threadIdx.x);
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

// Dynamic LDS of a lane-pair workgroup so that at most `per_cu` of them
// share a CU.
static size_t lp_lds_reserve(int per_cu) {
  const size_t cu = (size_t)cu_lds_bytes();
  const size_t want = per_cu == 1 ? cu / 2 + 4096 : cu / 2 - 1024;
  return want > sizeof(LpLds) ? want - sizeof(LpLds) : 0;
}

// Lane-pair workgroups per CU for a batch of n requests: the lane-pair
// kernel shortens every chain but needs three waves per 64 requests, so it
// runs while the batch fits in one or two workgroups per CU (latency-bound
// batches); larger batches keep every SIMD busy with the single-wave kernel
// (0).
static int lp_slots(int32_t n) {
  if (n <= 0) return 0;
  const int64_t groups = ceil_div(n, (int64_t)kWave);
  const int64_t cus = device_cu_count();
  if (groups <= cus) return 1;
  if (groups <= 2 * cus) return 2;
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

int stream_scratch(hipStream_t s, size_t bytes, void **ptr, std::unique_lock<std::mutex> &lk) {
  static std::mutex mu;
  // keyed by device and stream; hipStreamPerThread names a different stream
  // in every host thread, so the thread is part of its key
  using Key = std::tuple<int, hipStream_t, std::thread::id>;
  static std::map<Key, std::pair<void *, size_t>> bufs;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return KVGOV_E_HIP;
  const std::thread::id tid =
      s == hipStreamPerThread ? std::this_thread::get_id() : std::thread::id();
  lk = std::unique_lock<std::mutex>(mu);
  std::pair<void *, size_t> &b = bufs[Key(dev, s, tid)];
  if (b.second < bytes) {
    constexpr size_t kGrain = 64 * 1024;
    const size_t cap = (std::max(bytes, 2 * b.second) + kGrain - 1) / kGrain * kGrain;
    if (b.first) {
      // earlier calls on s may still read the old buffer
      const bool ok = hipStreamSynchronize(s) == hipSuccess && hipFree(b.first) == hipSuccess;
      b = {nullptr, 0};
      if (!ok) {
        lk.unlock();
        return KVGOV_E_HIP;
      }
    }
    void *p = nullptr;
    if (hipMalloc(&p, cap) != hipSuccess) {
      (void)hipGetLastError();  // not left for the next launch check
      lk.unlock();
      return KVGOV_E_NOMEM;
    }
    b = {p, cap};
  }
  *ptr = b.first;
  return KVGOV_OK;
}

// Scratch of the allocation-free hashing entry point: the longest-first
// order of a batch (histogram, then the order), kOrderBuckets + n int32 for
// n up to KVGOV_NOALLOC_MAX_REQUESTS.  One copy per device, held until the
// process ends; host code reaches it only through the address that
// hipGetSymbolAddress returns on that device (the array's name is a host
// stand-in, not a device address).
constexpr int64_t kNoAllocScratchInts = (int64_t)kOrderBuckets + KVGOV_NOALLOC_MAX_REQUESTS;
static __device__ __align__(256) int32_t scratch[kNoAllocScratchInts];

// Device address of `scratch` on the current device, looked up once per
// device; NULL if the lookup fails.
static int32_t *noalloc_scratch() {
  static std::mutex mu;
  static std::vector<int32_t *> ptrs;
  static std::vector<char> looked_up;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return nullptr;
  std::lock_guard<std::mutex> g(mu);
  if ((int)ptrs.size() <= dev) {
    ptrs.resize(dev + 1, nullptr);
    looked_up.resize(dev + 1, 0);
  }
  if (!looked_up[dev]) {
    int32_t *ptr = nullptr;
    if (hipGetSymbolAddress(reinterpret_cast<void **>(&ptr), HIP_SYMBOL(scratch)) != hipSuccess)
      return nullptr;  // not cached: a later call tries again
    ptrs[dev] = ptr;
    looked_up[dev] = 1;
  }
  return ptrs[dev];
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
    case KVGOV_E_INTERNAL:
      return "internal invariant failed inside a kernel (bounded wait or scratch contents)";
    case KVGOV_E_TOO_LARGE:
      return "batch above KVGOV_NOALLOC_MAX_REQUESTS requests (allocation-free entry point)";
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

static int block_offsets_impl(const int64_t *tok_offsets, const int32_t *start, int32_t n,
                              int32_t block_size, int64_t *blk_offsets, int32_t *status,
                              void *stream) {
  if (!tok_offsets || !blk_offsets || !status || n < 0) return KVGOV_E_INVAL;
  if (block_size != KVGOV_BLOCK_SIZE) return KVGOV_E_UNSUPPORTED;
  hipStream_t s = as_stream(stream);
  const int64_t tiles = std::max<int64_t>(1, ceil_div(n, kScanTile));
  std::unique_lock<std::mutex> lk;
  void *scratch_p = nullptr;
  const int src = stream_scratch(s, (size_t)tiles * sizeof(int64_t), &scratch_p, lk);
  if (src != KVGOV_OK) return src;
  int64_t *partial = static_cast<int64_t *>(scratch_p);
  hipLaunchKernelGGL(k_blk_partial, dim3((unsigned)tiles), dim3(kScanThreads), 0, s,
                     tok_offsets, start, n, partial, status);
  hipLaunchKernelGGL(k_blk_scan_partials, dim3(1), dim3(kScanThreads), 0, s, partial, tiles);
  hipLaunchKernelGGL(k_blk_write, dim3((unsigned)tiles), dim3(kScanThreads), 0, s, tok_offsets,
                     start, n, partial, blk_offsets, status);
  return launch_status();
}

int kvgov_block_offsets(const int64_t *tok_offsets, int32_t n, int32_t block_size,
                        int64_t *blk_offsets, int32_t *status, void *stream) {
  return block_offsets_impl(tok_offsets, nullptr, n, block_size, blk_offsets, status, stream);
}

int kvgov_resume_offsets(const int64_t *tok_offsets, const int32_t *start_block, int32_t n,
                         int32_t block_size, int64_t *blk_offsets, int32_t *status,
                         void *stream) {
  if (n > 0 && !start_block) return KVGOV_E_INVAL;
  return block_offsets_impl(tok_offsets, start_block, n, block_size, blk_offsets, status, stream);
}

// Longest-first order of a batch's requests (counting sort of their block
// counts) in `buf`: kOrderBuckets + n int32 (the histogram, then the
// order).  Returns the order.
static const int32_t *order_requests(const int64_t *blk_offsets, int32_t n, int32_t *buf,
                                     int32_t *status, hipStream_t s) {
  int32_t *hist = buf;
  int32_t *order = buf + kOrderBuckets;
  hipLaunchKernelGGL(k_fill_i32, dim3(kOrderBuckets / 256), dim3(256), 0, s, hist,
                     (int64_t)kOrderBuckets, 0);
  const dim3 tiles((unsigned)ceil_div(n, kOrderTile));
  hipLaunchKernelGGL(k_order_hist, tiles, dim3(kOrderThreads), 0, s, blk_offsets, n, hist);
  hipLaunchKernelGGL(k_order_scan, dim3(1), dim3(256), 0, s, hist);
  hipLaunchKernelGGL(k_order_scatter, tiles, dim3(kOrderThreads), 0, s, blk_offsets, n, hist,
                     order, status);
  return order;
}

// Events the next chain call of this host thread records around its chain
// kernel (kvgov_time_next_chain_kernel); taken and cleared by that call.
static thread_local hipEvent_t t_chain_events[2] = {nullptr, nullptr};

static int hash_chains_impl(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_offsets,
                            int32_t n, const int32_t *principal, const uint8_t *salts, int32_t P,
                            int32_t mode, const int32_t *boundary_tok, int32_t block_size,
                            const int32_t *start, const uint8_t *parents,
                            const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                            int32_t *status, void *stream, bool noalloc) {
  const hipEvent_t ev_start = t_chain_events[0], ev_end = t_chain_events[1];
  t_chain_events[0] = t_chain_events[1] = nullptr;
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
  a.start = start;
  a.parents = parents;

  // Launch shape.  A chain wave is bound by its SIMD's issue rate, so it
  // should never share a SIMD while others sit idle.  The dispatcher stacks
  // the waves of concurrent launches on the same SIMDs, and the older wave
  // then takes nearly every issue slot, so the workgroups reserve LDS (unused
  // beyond the kernel's own) to bound how many share a CU.
  const int slots = lp_slots(n);
  std::unique_lock<std::mutex> lk;  // held while the ordered launch is enqueued
  if (slots) {
    // lane pairs: two rounds waves and a schedule wave per 64 requests, one
    // or two workgroups per CU; every request of the batch is resident from
    // the start, so the order of the requests does not matter
    // (one workgroup per CU: a fourth wave, which shares the schedule;
    // two: three waves, the schedule on one)
    const dim3 grid((unsigned)ceil_div(n, kWave));
    const size_t lds = lp_lds_reserve(slots);
    if (ev_start && hipEventRecord(ev_start, s) != hipSuccess) return KVGOV_E_HIP;
    if (slots == 1) {
      const dim3 block(4 * kWave);
      switch (mode) {
        case KVGOV_NONE: hipLaunchKernelGGL((k_chains_lp<KVGOV_NONE, true>), grid, block, lds, s, a); break;
        case KVGOV_ROOT: hipLaunchKernelGGL((k_chains_lp<KVGOV_ROOT, true>), grid, block, lds, s, a); break;
        default: hipLaunchKernelGGL((k_chains_lp<KVGOV_BOUNDARY, true>), grid, block, lds, s, a); break;
      }
    } else {
      const dim3 block(kLpThreads);
      switch (mode) {
        case KVGOV_NONE: hipLaunchKernelGGL((k_chains_lp<KVGOV_NONE, false>), grid, block, lds, s, a); break;
        case KVGOV_ROOT: hipLaunchKernelGGL((k_chains_lp<KVGOV_ROOT, false>), grid, block, lds, s, a); break;
        default: hipLaunchKernelGGL((k_chains_lp<KVGOV_BOUNDARY, false>), grid, block, lds, s, a); break;
      }
    }
  } else {
    // More than two lane-pair workgroups per CU: the batch has at least as
    // many waves (one lane per request) as the chip has SIMDs, and it is
    // ordered longest first (counting sort of block counts).  The longest
    // requests then run on lane-pair workgroups (one eighth of the CUs), the
    // rest one lane per request; one workgroup per CU.
    // The ordering scratch: the library's fixed array for the
    // allocation-free entry point, else the stream's own scratch.
    int32_t *buf = nullptr;
    if (noalloc) {
      buf = noalloc_scratch();
      if (!buf) return KVGOV_E_HIP;
    } else {
      const size_t bytes = sizeof(int32_t) * ((size_t)kOrderBuckets + (size_t)n);
      void *p = nullptr;
      const int src = stream_scratch(s, bytes, &p, lk);
      if (src != KVGOV_OK) return src;
      buf = static_cast<int32_t *>(p);
    }
    a.order = order_requests(blk_offsets, n, buf, status, s);
    const int32_t lp_groups = std::max(1, device_cu_count() / 8);
    const int64_t rest = std::max<int64_t>(0, (int64_t)n - (int64_t)lp_groups * kWave);
    const dim3 grid((unsigned)(lp_groups + ceil_div(rest, 4 * kWave))), block(4 * kWave);
    const size_t res = chain_lds_reserve();
    const size_t lds = res > sizeof(LpLds) ? res - sizeof(LpLds) : 0;
    if (ev_start && hipEventRecord(ev_start, s) != hipSuccess) return KVGOV_E_HIP;
    switch (mode) {
      case KVGOV_NONE: hipLaunchKernelGGL(k_chains_mixed<KVGOV_NONE>, grid, block, lds, s, a, lp_groups); break;
      case KVGOV_ROOT: hipLaunchKernelGGL(k_chains_mixed<KVGOV_ROOT>, grid, block, lds, s, a, lp_groups); break;
      default: hipLaunchKernelGGL(k_chains_mixed<KVGOV_BOUNDARY>, grid, block, lds, s, a, lp_groups); break;
    }
  }
  int rc = launch_status();
  if (ev_end && hipEventRecord(ev_end, s) != hipSuccess && rc == KVGOV_OK) rc = KVGOV_E_HIP;
  return rc;
}

int kvgov_time_next_chain_kernel(void *start_event, void *end_event) {
  if ((start_event == nullptr) != (end_event == nullptr)) return KVGOV_E_INVAL;
  t_chain_events[0] = static_cast<hipEvent_t>(start_event);
  t_chain_events[1] = static_cast<hipEvent_t>(end_event);
  return KVGOV_OK;
}

int kvgov_hash_chains(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_offsets,
                      int32_t n, const int32_t *principal, const uint8_t *salts, int32_t P,
                      int32_t mode, const int32_t *boundary_tok, int32_t block_size,
                      const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                      int32_t *status, void *stream) {
  return hash_chains_impl(tokens, n_tokens, tok_offsets, n, principal, salts, P, mode,
                          boundary_tok, block_size, nullptr, nullptr, blk_offsets, hashes,
                          n_blocks, status, stream, false);
}

int kvgov_hash_chains_noalloc(const int32_t *tokens, int64_t n_tokens,
                              const int64_t *tok_offsets, int32_t n, const int32_t *principal,
                              const uint8_t *salts, int32_t P, int32_t mode,
                              const int32_t *boundary_tok, int32_t block_size,
                              const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                              int32_t *status, void *stream) {
  if (n > KVGOV_NOALLOC_MAX_REQUESTS) return KVGOV_E_TOO_LARGE;
  return hash_chains_impl(tokens, n_tokens, tok_offsets, n, principal, salts, P, mode,
                          boundary_tok, block_size, nullptr, nullptr, blk_offsets, hashes,
                          n_blocks, status, stream, true);
}

int kvgov_hash_chains_resume(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_offsets,
                             int32_t n, const int32_t *principal, const uint8_t *salts,
                             int32_t P, int32_t mode, const int32_t *boundary_tok,
                             int32_t block_size, const int32_t *start_block,
                             const uint8_t *parents, const int64_t *blk_offsets, uint8_t *hashes,
                             int64_t n_blocks, int32_t *status, void *stream) {
  if (n > 0 && (!start_block || !parents)) return KVGOV_E_INVAL;
  if (reinterpret_cast<uintptr_t>(parents) & 3) return KVGOV_E_INVAL;
  return hash_chains_impl(tokens, n_tokens, tok_offsets, n, principal, salts, P, mode,
                          boundary_tok, block_size, start_block, parents, blk_offsets, hashes,
                          n_blocks, status, stream, false);
}

}  // extern "C"
