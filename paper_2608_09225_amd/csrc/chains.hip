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

template <int MODE>
__global__ __launch_bounds__(256) void k_chains(ChainArgs a) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int32_t r = a.order ? a.order[i] : i;

  // ---- validate this request; a rejected request writes nothing
  const int64_t t0 = a.tok_offsets[r], t1 = a.tok_offsets[r + 1];
  if (t0 < 0 || t1 < t0 || t1 > a.n_tokens) {
    latch(a.status, KVGOV_E_OFFSETS);
    return;
  }
  const int64_t len = t1 - t0;
  const int64_t nf = len >> 4;
  const int64_t b0 = a.blk_offsets[r];
  if (b0 < 0 || a.blk_offsets[r + 1] - b0 != nf || b0 + nf > a.n_blocks) {
    latch(a.status, KVGOV_E_OFFSETS);
    return;
  }
  uint32_t sig[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (MODE != KVGOV_NONE) {
    const int32_t p = a.principal[r];
    if (p < 0 || p >= a.P) {
      latch(a.status, KVGOV_E_PRINCIPAL);
      return;
    }
    load_digest(a.salts + (int64_t)p * 32, sig);
  }
  int64_t k = -1;  // salted block (boundary mode)
  if (MODE == KVGOV_BOUNDARY) {
    const int32_t bt = a.boundary_tok[r];
    if (bt < 0 || bt > len) {
      latch(a.status, KVGOV_E_BOUNDARY);
      return;
    }
    k = bt >> 4;
  }
  if (nf == 0) return;

  const int32_t *tp = a.tokens + t0;
  uint8_t *out = a.hashes + b0 * 32;

  // H holds h_{j-1} as state words; a root-salted first block (and k == 0 in
  // boundary mode) is the usual pattern with sigma in place of h_{-1}.
  uint32_t H[8];
  const bool salted_root = (MODE == KVGOV_ROOT) || (MODE == KVGOV_BOUNDARY && k == 0);
#pragma unroll
  for (int q = 0; q < 8; ++q) H[q] = salted_root ? sig[q] : 0u;

  u32x4 nxt[4];
  load_raw(tp, nxt);
  // special-path flags: unsalted 64-byte first block, boundary block
  const bool plain_first = !salted_root;

  for (int64_t j = 0; j < nf; ++j) {
    uint32_t T[16];
    swap_block(nxt, T);
    if (j + 1 < nf) load_raw(tp + 16 * (j + 1), nxt);

    const bool u0 = plain_first && j == 0;
    const bool bnd = (MODE == KVGOV_BOUNDARY) && j == k && k > 0;
    uint32_t st[8], w[16];
    if (MODE == KVGOV_ROOT || !__any(u0 || bnd)) {
      // hot path: (IV; h || T[0..7]) then (state; T[8..15] || pad96)
      set_iv(st);
#pragma unroll
      for (int q = 0; q < 8; ++q) { w[q] = H[q]; w[8 + q] = T[q]; }
      compress(st, w);
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = T[8 + q];
      w[8] = 0x80000000u;
#pragma unroll
      for (int q = 9; q < 15; ++q) w[q] = 0;
      w[15] = 96 * 8;
      compress(st, w);
    } else {
      // special path, per lane:
      //   normal  : (IV; h || T[0..7])        (state; T[8..15] || pad96)
      //   u0      : (IV; T[0..15])            (state; pad64)
      //   boundary: (IV; sigma || h) -> X,   (X; T[0..15])   (state; pad128)
      uint32_t X[8];
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
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) H[q] = st[q];
    store_digest(out + j * 32, H);
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
// and the kernel takes as long as its longest chain in any order.
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

  int32_t *scratch = nullptr;
  if (n >= order_min_requests()) {
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
  // then takes nearly every issue slot, so the workgroup reserves more than
  // half of a CU's LDS (unused by the kernel): at most one chain workgroup
  // per CU.  Batches of at most one wave per CU run one wave per workgroup
  // (one SIMD per CU busy, every CU used); larger ones run four waves per
  // workgroup, one per SIMD.
  const int threads = (int64_t)n <= (int64_t)device_cu_count() * kWave ? kWave : 4 * kWave;
  const dim3 grid((unsigned)ceil_div(n, threads)), block(threads);
  const size_t lds = chain_lds_reserve();
  switch (mode) {
    case KVGOV_NONE: hipLaunchKernelGGL(k_chains<KVGOV_NONE>, grid, block, lds, s, a); break;
    case KVGOV_ROOT: hipLaunchKernelGGL(k_chains<KVGOV_ROOT>, grid, block, lds, s, a); break;
    default: hipLaunchKernelGGL(k_chains<KVGOV_BOUNDARY>, grid, block, lds, s, a); break;
  }
  int rc = launch_status();
  if (scratch && hipFreeAsync(scratch, s) != hipSuccess && rc == KVGOV_OK) rc = KVGOV_E_HIP;
  return rc;
}

}  // extern "C"
