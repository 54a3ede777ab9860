// Device-resident prefix-cache table: batched insert and first-miss lookup.
//
// Paper: a block prefix cache keys KV blocks by their chained block hash and
// resolves a request to the longest cached prefix, quantised to blocks; the
// prober learns the number of leading blocks matched (Sec. 2.1; Table
// tab:taxonomy, block prefix cache row).
//
// Layout (HBM):
//   keys [slots][32 B]  the stored keys; an empty slot holds 32 bytes 0xFF.
//                       Lookups read only this array: a probe is one 32-byte
//                       read, and a probe sequence runs through the four
//                       slots of its 128-byte line before it leaves it.
//   tags [slots] u64    0 = empty, else (epoch << 32) | (claimant + 1): the
//                       insert call that claimed the slot and the index of the
//                       claiming key within that call's input.
//   meta                key count, per-call counters, latched error, and the
//                       tag and presence bit of the all-0xFF key, which cannot
//                       live in a slot because it is the empty pattern.
//
// Insert protocol (no fences, no waiting on other lanes).  A key walks its
// probe sequence; at each slot it reads the tag:
//   * empty          -> CAS the tag to (epoch, me); the winner writes the key
//                       into the slot and counts one new key.
//   * earlier epoch  -> the slot's key was written by an earlier kernel and is
//                       visible: compare all 256 bits.
//   * current epoch  -> the slot was claimed in this call; its key may not be
//                       written yet, so compare against the claimant's key in
//                       this call's input array instead.
// Equal -> already present, stop.  Otherwise move to the next slot.  Two
// copies of one key follow the same sequence and each slot changes state at
// most once, so exactly one copy claims a slot and the other finds it.
//
// Admission (lookup-then-insert in request order) runs the same insert and
// additionally lowers a slot claimed in the call to the smallest claiming
// row (atomicMin on the tag: the epoch bits are equal, so the minimum is the
// earliest row, i.e. the earliest request holding the key), and records per
// row which slot its key went to; a second kernel then decides per request
// what it sees: keys of earlier calls, and keys whose earliest row lies in an
// earlier request.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <new>

#include "table.h"

namespace kvgov {

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_cache_fill(u32x4 *keys, unsigned long long *tags,
                                                    unsigned long long *rank, int64_t slots,
                                                    CacheMeta *m) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  const u32x4 ones = u32x4{0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < kCounterLanes; i += blockDim.x) {
      m->n_keys[i] = 0;
      m->new_keys[0][i] = 0;
      m->new_keys[1][i] = 0;
    }
    if (threadIdx.x == 0) {
      m->exported = 0;
      m->ones_tag = 0;
      m->ones_rank = 0;
      m->status = 0;
      m->ones_present = 0;
    }
  }
  for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < slots; s += stride) {
    keys[2 * s] = ones;
    keys[2 * s + 1] = ones;
    tags[s] = 0;
    if (rank) rank[s] = 0;
  }
}

// Consecutive keys per wave chunk of k_chunk_insert.  Longer chunks mean fewer
// waves in flight at once, so that the copies of a key that many requests
// hold (a principal's shared prefix) reach its slot over a longer span and
// most of them find it claimed by a plain read instead of racing for it
// with compare-and-swaps on one address (measured: 256 beats 64, 128, 512).
constexpr int kInsChunk = 256;

// The largest r in [0, n) with bo[r] <= f (bo non-decreasing in a valid
// batch; any answer in range is harmless otherwise, see k_chunk_insert).  Every
// lane of a wave searches the same f.
__device__ __forceinline__ int32_t find_request(const int64_t *bo, int32_t n, int64_t f) {
  int32_t a = 0, b = n - 1;
  while (a < b) {
    const int32_t mid = (a + b + 1) >> 1;
    if (bo[mid] <= f) a = mid; else b = mid - 1;
  }
  return a;
}

// Insert walking the batch in chunks of kInsChunk consecutive rows per wave,
// 64 at a time: the admission's first half (ADMIT), and the plain insert of
// batches whose requests are so long that a group per request would leave
// the chip idle (a flat key set given as one request).  Before touching the
// table a key is compared with the key at the same block position of the
// previous request (requests that share a prefix - the same principal, or
// any principal below the boundary block - hold the same keys there): an
// equal earlier key makes this one a duplicate that needs no table access,
// so a prefix shared by thousands of requests costs a few table operations
// per key instead of thousands of atomics on one slot.  The request of each
// key comes from a window of 64 request starts (a search over lanes); the
// comparison is only an optimisation: skipping a key that equals an
// earlier key of the batch is always correct (the earlier one is inserted,
// or is itself a duplicate of an earlier one), and the compared position
// is checked to lie in the batch, so malformed interior offsets cannot
// cause a wrong result or an out-of-range read.  A row's request, and so
// its depth (its position in the request, which the recency rank holds),
// is exact: rows whose request lies past the window search for it.
//
// ADMIT: claims are lowered to the earliest row, and codes[f] records where
// row f's key went (kCodeDup for a key skipped as equal to the previous
// request's, which is in an earlier request by construction).
template <bool ADMIT>
__global__ __launch_bounds__(256) void k_chunk_insert(TableView t, const uint8_t *hashes,
                                                      const int64_t *blk_offsets, int32_t n,
                                                      int64_t n_blocks, uint32_t epoch,
                                                      uint32_t *codes) {
  __shared__ uint32_t lds4[4];
  const int64_t lo = blk_offsets[0], hi = blk_offsets[n];
  const bool first = blockIdx.x == 0 && threadIdx.x == 0;
  if (blockIdx.x == 0 && threadIdx.x < kCounterLanes)
    t.meta->new_keys[(epoch + 1) & 1][threadIdx.x] = 0;  // counters of the next call
  if (lo < 0 || hi < lo || hi > n_blocks || hi - lo >= 0xFFFFFFFFll) {
    if (first) atomicCAS(&t.meta->status, 0, KVGOV_E_OFFSETS);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * 4;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  uint32_t added = 0;
  for (int64_t f0 = lo + wave * kInsChunk; f0 < hi; f0 += waves * kInsChunk) {
    const int64_t f1 = f0 + kInsChunk < hi ? f0 + kInsChunk : hi;
    int32_t rc = find_request(blk_offsets, n, f0);
    for (int64_t fb = f0; fb < f1; fb += 64) {
      // win[l] = start of request rc - 1 + l (clamped to [0, n])
      int32_t wi = rc - 1 + lane;
      wi = wi < 0 ? 0 : (wi > n ? n : wi);
      const int64_t win = blk_offsets[wi];
      const int64_t f = fb + lane;
      // pos: the largest l in [1, 63] with win[l] <= f
      int pos = 1;
#pragma unroll
      for (int step = 32; step >= 1; step >>= 1) {
        const int cand = pos + step;
        const int64_t v = __shfl(win, cand < 63 ? cand : 63, 64);
        if (cand <= 63 && v <= f) pos = cand;
      }
      int64_t b_r = __shfl(win, pos, 64);
      int64_t b_p = __shfl(win, pos - 1, 64);
      int32_t r = rc - 1 + pos;
      if (pos == 63) {
        // 64 rows can span more requests than the window reaches (requests
        // of one block or none): a row whose request starts past the window
        // finds it by binary search (its depth depends on it)
        const int32_t ne = rc + 63;
        if (ne < n && blk_offsets[ne] <= f) {
          r = find_request(blk_offsets, n, f);
          b_r = blk_offsets[r];
          b_p = blk_offsets[r - 1];
        }
      }
      if (f < f1) {
        const Key key = load_key(hashes + f * 32);
        bool dup = false;
        const int64_t jj = f - b_r;
        if (r >= 1 && jj >= 0 && jj < b_r - b_p && b_p + jj >= lo)
          dup = key_eq(key, load_key(hashes + (b_p + jj) * 32));
        uint32_t code = kCodeDup;
        // the depth of the key: its row within its request (clamped; only
        // malformed interior offsets put it outside [0, 2^31))
        const uint32_t depth = (uint32_t)(jj < 0 ? 0 : (jj > 0x7FFFFFFF ? 0x7FFFFFFF : jj));
        if (!dup) added += insert_key<ADMIT>(t, key, f, lo, hashes, epoch, &code, depth);
        if (ADMIT) codes[f] = code;
      }
      rc = __shfl(r, 63, 64);
    }
  }
  const uint32_t total = block_sum(added, lds4);
  if (threadIdx.x == 0 && total) {
    const int cl = blockIdx.x % kCounterLanes;
    atomicAdd(&t.meta->new_keys[epoch & 1][cl], (unsigned long long)total);
    atomicAdd(&t.meta->n_keys[cl], (unsigned long long)total);
  }
}

// Plain (set-union) insert with G lanes per request, which walk the
// request's rows G at a time.  Two comparisons keep keys that many requests
// share away from the table (a key skipped by either equals a row of the
// batch that lies before it, and the earliest row of any key is never
// skipped, so every key reaches the table):
//   * the previous request's row at the same depth (requests that share a
//     prefix and are adjacent, e.g. a prefix below the boundary block that
//     every request holds);
//   * the row at the same depth of an earlier request that starts with the
//     same key: the group's first lane inserts the request's first row
//     before the others start, and if the slot's tag names an earlier row
//     (the request that claimed the key, mostly the earliest one, since
//     workgroups start in request order) the group compares against the
//     rows that follow it.  Requests of one principal share the
//     root-salted prefix but are rarely adjacent.  (Lowering the tag to the
//     earliest first row with an atomic minimum, as admission does, measured
//     slower: 35.7 -> 36.6 us for the paper-shaped root-mode insert.)
// On a table that tracks recency only the first comparison is made (the
// second one's row may lie past the end of that request, at another depth,
// and a key's rank holds its smallest depth).
// Each request inserts the rows [blk_offsets[r], blk_offsets[r + 1]) cut to
// the batch [blk_offsets[0], blk_offsets[n]); requests whose offsets are out
// of order insert nothing.  With non-decreasing offsets that is every row
// once.  Otherwise every row of the batch still lies in some request's
// range (take the last r with blk_offsets[r] <= row), so the table receives
// exactly the batch's keys.
template <int G>
__global__ __launch_bounds__(256) void k_insert_req(TableView t, const uint8_t *hashes,
                                                    const int64_t *blk_offsets, int32_t n,
                                                    int64_t n_blocks, uint32_t epoch) {
  __shared__ uint32_t lds4[4];
  const int64_t lo = blk_offsets[0], hi = blk_offsets[n];
  if (blockIdx.x == 0 && threadIdx.x < kCounterLanes)
    t.meta->new_keys[(epoch + 1) & 1][threadIdx.x] = 0;  // counters of the next call
  if (lo < 0 || hi < lo || hi > n_blocks || hi - lo >= 0xFFFFFFFFll) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicCAS(&t.meta->status, 0, KVGOV_E_OFFSETS);
    return;
  }
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t r = gid / G;
  const int sub = (int)(gid % G);
  const int lane = threadIdx.x & 63;
  const int base = lane & ~(G - 1);
  uint32_t added = 0;
  // groups never straddle r < n (256 % G == 0); the block sum below needs
  // every thread, so out-of-range groups only skip the work
  if (r < n) {
    const int64_t b_r = blk_offsets[r], b_e = blk_offsets[r + 1];
    const int64_t b_p = r >= 1 ? blk_offsets[r - 1] : 0;
    const int64_t b0 = b_r > lo ? b_r : lo, b1 = b_e < hi ? b_e : hi;
    // the previous request's rows, when its range is in order and in the batch
    const int64_t n_p = r >= 1 && b_p >= lo && b_p <= b_r ? b_r - b_p : 0;
    if (b0 < b1) {
      // first row, by the group's first lane
      int64_t g0 = -1;
      if (sub == 0) {
        const int64_t jj = b0 - b_r;
        const Key key = load_key(hashes + b0 * 32);
        const bool dup = jj < n_p && key_eq(key, load_key(hashes + (b_p + jj) * 32));
        if (!dup) {
          uint32_t code;
          unsigned long long claim = 0;
          added += insert_key<false>(t, key, b0, lo, hashes, epoch, &code, (uint32_t)jj, &claim);
          const int64_t c = lo + (int64_t)(claim & 0xFFFFFFFFull) - 1;
          if (!t.track && jj == 0 && (uint32_t)(claim >> 32) == epoch && c >= lo && c < b0)
            g0 = c;
        }
      }
      g0 = __shfl(g0, base, 64);
      for (int64_t f = b0 + 1 + sub; f < b1; f += G) {
        const int64_t jj = f - b_r;
        const Key key = load_key(hashes + f * 32);
        bool dup = jj < n_p && key_eq(key, load_key(hashes + (b_p + jj) * 32));
        if (!dup && g0 >= 0) dup = key_eq(key, load_key(hashes + (g0 + jj) * 32));
        uint32_t code;
        const uint32_t depth = (uint32_t)(jj > 0x7FFFFFFF ? 0x7FFFFFFF : jj);
        if (!dup) added += insert_key<false>(t, key, f, lo, hashes, epoch, &code, depth);
      }
    }
  }
  const uint32_t total = block_sum(added, lds4);
  if (threadIdx.x == 0 && total) {
    const int cl = blockIdx.x % kCounterLanes;
    atomicAdd(&t.meta->new_keys[epoch & 1][cl], (unsigned long long)total);
    atomicAdd(&t.meta->n_keys[cl], (unsigned long long)total);
  }
}

struct LookupArgs {
  TableView t;
  const uint8_t *hashes;
  const int64_t *blk_offsets;
  int32_t n;
  int64_t n_blocks;
  int32_t *hit_blocks;
};

// G lanes per request take G consecutive blocks at a time; a ballot over the
// group finds the first miss, and the group stops at the first chunk that
// holds one.  Several probes in flight per lane (over blocks past the first
// miss: 2 or 4 per lane) measured slower on the probe-heavy workload, whose
// lookup is bound by the lines it moves rather than by latency.
template <int G>
__global__ __launch_bounds__(256) void k_lookup(LookupArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t r = gid / G;
  if (r >= a.n) return;  // groups never straddle this test: 256 % G == 0
  const int sub = (int)(gid % G);
  const int lane = threadIdx.x & 63;
  const int base = lane & ~(G - 1);
  const uint64_t gmask = group_mask<G>(base);
  const int64_t b0 = a.blk_offsets[r], b1 = a.blk_offsets[r + 1];
  if (b0 < 0 || b1 < b0 || b1 > a.n_blocks) {
    if (sub == 0) {
      atomicCAS(&a.t.meta->status, 0, KVGOV_E_OFFSETS);
      a.hit_blocks[r] = 0;
    }
    return;
  }
  const bool ones = a.t.meta->ones_present != 0;
  const int64_t nf = b1 - b0;
  int64_t hit = nf;
  for (int64_t j0 = 0; j0 < nf; j0 += G) {
    const int64_t j = j0 + sub;
    bool miss = false;
    if (j < nf) miss = !probe(a.t, load_key(a.hashes + (b0 + j) * 32), ones);
    const uint64_t m = __ballot(miss) & gmask;
    if (m) {
      hit = j0 + (__builtin_ctzll(m) - base);
      break;
    }
  }
  if (sub == 0) a.hit_blocks[r] = (int32_t)hit;
}

struct AdmitArgs {
  TableView t;
  const int64_t *blk_offsets;
  int32_t n;
  int64_t n_blocks;
  uint32_t epoch;
  const uint32_t *codes;  // per row, from k_chunk_insert<true>
  int32_t *hit_blocks;
  int32_t *new_blocks;
};

// Second half of the admission: G lanes per request walk all of its rows G
// at a time.  Row f of request r (rows [b0, b1)) with key K:
//   visible to r  <=>  K was in the table before the call (a tag of an
//                      earlier epoch), or K's earliest row in the call lies
//                      before b0 (an earlier request holds it);
//   new for r     <=>  K's earliest row is f itself.
// hit_blocks[r] = first row not visible (relative to b0), new_blocks[r] =
// rows new for r.  The earliest rows are final: k_chunk_insert<true> has ended.
template <int G>
__global__ __launch_bounds__(256) void k_admit_scan(AdmitArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t r = gid / G;
  if (r >= a.n) return;  // groups never straddle this test: 256 % G == 0
  const int sub = (int)(gid % G);
  const int lane = threadIdx.x & 63;
  const int base = lane & ~(G - 1);
  const uint64_t gmask = group_mask<G>(base);
  const int64_t lo = a.blk_offsets[0], hi = a.blk_offsets[a.n];
  const int64_t b0 = a.blk_offsets[r], b1 = a.blk_offsets[r + 1];
  // the batch check of k_chunk_insert<true> (which then wrote no codes), and this
  // request's rows inside the batch
  if (lo < 0 || hi < lo || hi > a.n_blocks || hi - lo >= 0xFFFFFFFFll || b0 < lo || b1 < b0 ||
      b1 > hi) {
    if (sub == 0) {
      atomicCAS(&a.t.meta->status, 0, KVGOV_E_OFFSETS);
      a.hit_blocks[r] = 0;
      a.new_blocks[r] = 0;
    }
    return;
  }
  const int64_t nf = b1 - b0;
  int64_t hit = nf;
  uint32_t fresh = 0;
  for (int64_t j0 = 0; j0 < nf; j0 += G) {
    const int64_t j = j0 + sub;
    bool seen = true;
    if (j < nf) {
      const int64_t f = b0 + j;
      const uint32_t code = a.codes[f];
      if (code == kCodeFailed) {
        seen = false;
      } else if (code != kCodeDup) {
        const unsigned long long tag =
            code == kCodeOnes ? a.t.meta->ones_tag : a.t.tags[code];
        if ((uint32_t)(tag >> 32) == a.epoch) {
          const int64_t first = lo + (int64_t)(tag & 0xFFFFFFFFull) - 1;
          seen = first < b0;
          fresh += first == f ? 1u : 0u;
        }
      }
    }
    const uint64_t m = __ballot(!seen) & gmask;
    if (m && hit == nf) hit = j0 + (__builtin_ctzll(m) - base);
  }
  // sum of `fresh` over the group
#pragma unroll
  for (int d = G / 2; d >= 1; d >>= 1) fresh += __shfl_xor(fresh, d, 64);
  if (sub == 0) {
    a.hit_blocks[r] = (int32_t)hit;
    a.new_blocks[r] = (int32_t)fresh;
  }
}

__global__ void k_export_begin(CacheMeta *m) { m->exported = 0; }

// One atomic per wave reserves the output rows of the wave's keys.
__device__ __forceinline__ void export_key(bool have, const u32x4 &lo, const u32x4 &hi,
                                           CacheMeta *m, uint8_t *out, int64_t cap) {
  const uint64_t mask = __ballot(have);
  if (!mask) return;
  const int lane = threadIdx.x & 63;
  const int leader = __builtin_ctzll(mask);
  unsigned long long base = 0;
  if (lane == leader) base = atomicAdd(&m->exported, (unsigned long long)__popcll(mask));
  base = __shfl(base, leader, 64);
  if (have) {
    const int64_t at = (int64_t)base + __popcll(mask & ((1ull << lane) - 1ull));
    if (at < cap) {
      u32x4 *q = reinterpret_cast<u32x4 *>(out + at * 32);
      q[0] = lo;
      q[1] = hi;
    }
  }
}

__global__ __launch_bounds__(256) void k_export(TableView t, uint8_t *out, int64_t cap) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  const int64_t slots = (int64_t)t.mask + 1;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const u32x4 ones = u32x4{0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
  if (blockIdx.x == 0 && threadIdx.x < 64)
    export_key(threadIdx.x == 0 && t.meta->ones_present != 0, ones, ones, t.meta, out, cap);
  // every lane of a wave runs the same number of iterations (ballot inside)
  const int64_t rounds = (slots + stride - 1) / stride;
  for (int64_t k = 0; k < rounds; ++k) {
    const int64_t s = gid + k * stride;
    const bool have = s < slots && t.tags[s] != 0;
    u32x4 lo = ones, hi = ones;
    if (have) {
      lo = t.keys[2 * s];
      hi = t.keys[2 * s + 1];
    }
    export_key(have, lo, hi, t.meta, out, cap);
  }
}

// ---------------------------------------------------------------------------
// maintenance: eviction by recency rank, erase, and the rebuild both end in
// ---------------------------------------------------------------------------

// Eviction keeps every key whose recency word (newer stamp first, then
// smaller depth) is at least a threshold chosen by a radix select over the
// 64-bit words, 8 bits per pass.

struct SelectState {
  unsigned long long prefix;     // rank bits decided so far
  unsigned long long threshold;  // keep rank >= threshold once done
  long long budget;              // keys still allowed below the decided part
  unsigned long long kept;       // keys copied out by the compaction
  unsigned long long erased;     // keys marked by erase
  unsigned long long n_dense;    // recency words gathered for the select
  unsigned long long lo, hi;     // their minimum and maximum
  int32_t level;                 // 8-bit digits decided
  int32_t done;
};

constexpr int kRankBins = 256;
constexpr int kCompactItems = 16;  // slots per thread per block step

// Exclusive prefix of v over the workgroup (256 threads) and the total; one
// global atomic on `counter` per call reserves the workgroup's range, whose
// start is returned in *base.  Several hundred workgroups hitting one counter
// once per 4096 slots cost little; once per wave they serialised (~200 us
// for a 2^20-slot table).
__device__ __forceinline__ uint32_t block_reserve(uint32_t v, unsigned long long *counter,
                                                  unsigned long long *base) {
  __shared__ uint32_t wsum[4];
  __shared__ unsigned long long wbase;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t u = __shfl_up(inc, d, 64);
    if (lane >= d) inc += u;
  }
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  uint32_t before = 0, total = 0;
  for (int i = 0; i < 4; ++i) {
    before += i < w ? wsum[i] : 0u;
    total += wsum[i];
  }
  if (threadIdx.x == 0) wbase = total ? atomicAdd(counter, (unsigned long long)total) : 0ull;
  __syncthreads();
  *base = wbase;
  __syncthreads();  // wsum and wbase are reused by the next call
  return before + inc - v;
}

// Gathers the recency words of the occupied slots (and of the all-0xFF key)
// into a dense array: the select passes then read 8 bytes per key instead
// of 16 per slot.
__global__ __launch_bounds__(256) void k_gather_ranks(TableView t, SelectState *st,
                                                      unsigned long long *dense) {
  const int64_t slots = (int64_t)t.mask + 1;
  const int64_t step = (int64_t)256 * kCompactItems;
  for (int64_t b0 = (int64_t)blockIdx.x * step; b0 < slots; b0 += (int64_t)gridDim.x * step) {
    unsigned long long r[kCompactItems];
    uint32_t have = 0;
#pragma unroll
    for (int k = 0; k < kCompactItems; ++k) {
      const int64_t s = b0 + (int64_t)k * 256 + threadIdx.x;
      r[k] = 0;
      if (s < slots && t.tags[s] != 0) {
        r[k] = t.rank[s];
        have |= 1u << k;
      }
    }
    unsigned long long base;
    uint32_t at = block_reserve(__popc(have), &st->n_dense, &base);
    unsigned long long mn = ~0ull, mx = 0;
#pragma unroll
    for (int k = 0; k < kCompactItems; ++k) {
      if (have & (1u << k)) {
        dense[base + at++] = r[k];
        mn = r[k] < mn ? r[k] : mn;
        mx = r[k] > mx ? r[k] : mx;
      }
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      const unsigned long long a = __shfl_xor(mn, d, 64), b = __shfl_xor(mx, d, 64);
      mn = a < mn ? a : mn;
      mx = b > mx ? b : mx;
    }
    // a wave holding keys reports its range even when every word is 0 (keys
    // inserted while tracking was off): the select must see that class too
    const bool any = __ballot(have != 0) != 0;
    if ((threadIdx.x & 63) == 0 && any) {
      atomicMin(&st->lo, mn);
      atomicMax(&st->hi, mx);
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && t.meta->ones_present) {
    const unsigned long long r = t.meta->ones_rank;
    dense[atomicAdd(&st->n_dense, 1ull)] = r;
    atomicMin(&st->lo, r);
    atomicMax(&st->hi, r);
  }
}

// Starts the select below the leading digits that all gathered words share
// (typically the high bytes of the stamp and of the depth), or ends it when
// they form one class.
__global__ void k_select_start(SelectState *st) {
  if (st->n_dense == 0) {
    st->done = 1;
    return;
  }
  const unsigned long long lo = st->lo, hi = st->hi;
  if (lo == hi) {
    st->threshold = st->n_dense <= (unsigned long long)st->budget ? 0ull : lo + 1;
    st->done = 1;
    return;
  }
  const int level = __builtin_clzll(lo ^ hi) / 8;  // 0..7
  st->level = level;
  st->prefix = level ? lo >> (64 - 8 * level) : 0ull;
}

// Histogram of the next digit of the gathered words that match the decided
// prefix, per workgroup in LDS.  Most keys of a table share the leading
// digits, so each wave first adds its lanes that share the first active
// lane's bin with one atomic.
__global__ __launch_bounds__(256) void k_rank_hist(const SelectState *st,
                                                   const unsigned long long *dense,
                                                   unsigned int *hist) {
  __shared__ unsigned int h[kRankBins];
  if (st->done) return;
  h[threadIdx.x] = 0;
  __syncthreads();
  const int level = st->level;
  const unsigned long long prefix = st->prefix;
  const int shift = 56 - 8 * level;
  const int64_t n = (int64_t)st->n_dense;
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * 256;
  // every lane of a wave runs the same number of rounds (ballot inside)
  const int64_t rounds = (n + stride - 1) / stride;
  for (int64_t k = 0; k < rounds; ++k) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x + k * stride;
    bool valid = false;
    int bin = 0;
    if (i < n) {
      const unsigned long long r = dense[i];
      valid = level == 0 || (r >> (shift + 8)) == prefix;
      bin = (int)((r >> shift) & 255);
    }
    const uint64_t act = __ballot(valid);
    if (!act) continue;
    const int leader = __builtin_ctzll(act);
    const int lbin = __shfl(bin, leader, 64);
    const uint64_t same = __ballot(valid && bin == lbin);
    if (lane == leader) atomicAdd(&h[lbin], (unsigned int)__popcll(same));
    if (valid && bin != lbin) atomicAdd(&h[bin], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&hist[threadIdx.x], h[threadIdx.x]);
}

// One workgroup: the digit at which the kept count crosses the budget (keys
// with a higher digit are kept), or the end when everything left fits.
// Leaves the histogram cleared for the next pass.
__global__ __launch_bounds__(256) void k_rank_select(SelectState *st, unsigned int *hist) {
  __shared__ unsigned long long c[kRankBins];
  __shared__ unsigned long long total;
  const int t = threadIdx.x;
  c[t] = hist[t];
  hist[t] = 0;
  const int done = st->done;
  const long long budget = st->budget;
  const int level = st->level;
  const unsigned long long prefix = st->prefix;
  __syncthreads();
  if (done) return;
  unsigned long long above = 0;  // keys whose digit exceeds t
  for (int u = t + 1; u < kRankBins; ++u) above += c[u];
  if (t == 0) total = above + c[0];
  __syncthreads();
  const unsigned long long B = (unsigned long long)budget;
  if (total <= B) {
    if (t == 0) {
      st->threshold = level == 0 ? 0ull : prefix << (64 - 8 * level);
      st->done = 1;
    }
    return;
  }
  if (above <= B && B < above + c[t]) {  // exactly one digit
    const unsigned long long p = (prefix << 8) | (unsigned long long)t;
    st->budget = budget - (long long)above;
    st->prefix = p;
    st->level = level + 1;
    if (level + 1 == 8) {  // the whole class p does not fit: keep what ranks above it
      st->threshold = p + 1;
      st->done = 1;
    }
  }
}

__global__ void k_select_init(SelectState *st, unsigned int *hist, long long budget,
                              int erase) {
  if (threadIdx.x == 0) {
    st->prefix = 0;
    st->threshold = 0;  // erase: keep every key not marked
    st->budget = budget;
    st->kept = 0;
    st->erased = 0;
    st->n_dense = 0;
    st->lo = ~0ull;
    st->hi = 0;
    st->level = 0;
    st->done = erase;
  }
  hist[threadIdx.x] = 0;
}

// Erase: a present key's recency word becomes kErased (counted once per key).
__global__ __launch_bounds__(256) void k_erase_mark(TableView t, const uint8_t *keys,
                                                    int64_t n, SelectState *st) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const Key k = load_key(keys + i * 32);
  unsigned long long *w = nullptr;
  if (key_is_empty_pattern(k)) {
    if (t.meta->ones_present) w = &t.meta->ones_rank;
  } else {
    const int64_t slot = find_slot(t, k);
    if (slot >= 0) w = &t.rank[slot];
  }
  if (w && atomicExch(w, kErased) != kErased) atomicAdd(&st->erased, 1ull);
}

// Copies the kept keys and their recency to scratch (one atomic per
// workgroup step of 4096 slots).
__global__ __launch_bounds__(256) void k_compact(TableView t, SelectState *st, u32x4 *out_keys,
                                                 unsigned long long *out_rank, int64_t cap) {
  const int64_t slots = (int64_t)t.mask + 1;
  const unsigned long long thr = st->threshold;
  const int64_t step = (int64_t)256 * kCompactItems;
  for (int64_t b0 = (int64_t)blockIdx.x * step; b0 < slots; b0 += (int64_t)gridDim.x * step) {
    uint32_t keep = 0;
#pragma unroll
    for (int k = 0; k < kCompactItems; ++k) {
      const int64_t s = b0 + (int64_t)k * 256 + threadIdx.x;
      if (s < slots && t.tags[s] != 0) {
        const unsigned long long r = t.rank[s];
        if (r != kErased && r >= thr) keep |= 1u << k;
      }
    }
    unsigned long long base;
    uint32_t at = block_reserve(__popc(keep), &st->kept, &base);
#pragma unroll
    for (int k = 0; k < kCompactItems; ++k) {
      if (!(keep & (1u << k))) continue;
      const int64_t s = b0 + (int64_t)k * 256 + threadIdx.x;
      const int64_t o = (int64_t)(base + at++);
      if (o < cap) {
        out_keys[2 * o] = t.keys[2 * s];
        out_keys[2 * o + 1] = t.keys[2 * s + 1];
        out_rank[o] = t.rank[s];
      }
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && t.meta->ones_present) {
    const unsigned long long r = t.meta->ones_rank;
    if (r != kErased && r >= thr) {
      const int64_t o = (int64_t)atomicAdd(&st->kept, 1ull);
      if (o < cap) {
        const u32x4 ones = u32x4{0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
        out_keys[2 * o] = ones;
        out_keys[2 * o + 1] = ones;
        out_rank[o] = r;
      }
    }
  }
}

// Empties the slots and the key counters for the rebuild; the latched error
// and the export count stay.
__global__ __launch_bounds__(256) void k_rebuild_fill(TableView t) {
  const int64_t slots = (int64_t)t.mask + 1;
  const u32x4 ones = u32x4{0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
  if (blockIdx.x == 0) {
    CacheMeta *m = t.meta;
    for (int i = threadIdx.x; i < kCounterLanes; i += blockDim.x) {
      m->n_keys[i] = 0;
      m->new_keys[0][i] = 0;
      m->new_keys[1][i] = 0;
    }
    if (threadIdx.x == 0) {
      m->ones_tag = 0;
      m->ones_rank = 0;
      m->ones_present = 0;
    }
  }
  for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < slots;
       s += (int64_t)gridDim.x * 256) {
    t.keys[2 * s] = ones;
    t.keys[2 * s + 1] = ones;
    t.tags[s] = 0;
    t.rank[s] = 0;
  }
}

// Inserts the kept keys again (all distinct) and restores their recency.
__global__ __launch_bounds__(256) void k_reinsert(TableView t, const SelectState *st,
                                                  const uint8_t *keys,
                                                  const unsigned long long *rank,
                                                  uint32_t epoch, int64_t cap) {
  __shared__ uint32_t lds4[4];
  int64_t n = (int64_t)st->kept;
  if (n > cap) {
    // more keys counted than the copy-out had room for (never expected: a
    // table holds at most cap keys): reinsert the copies only
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicCAS(&t.meta->status, 0, KVGOV_E_INTERNAL);
    n = cap;
  }
  uint32_t added = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256) {
    uint32_t code = kCodeFailed;
    added += insert_key<false>(t, load_key(keys + i * 32), i, 0, keys, epoch, &code);
    unsigned long long *dst =
        code == kCodeOnes ? &t.meta->ones_rank : (code < kCodeFailed ? &t.rank[code] : nullptr);
    if (dst) *dst = rank[i];
  }
  const uint32_t total = block_sum(added, lds4);
  if (threadIdx.x == 0 && total)
    atomicAdd(&t.meta->n_keys[blockIdx.x % kCounterLanes], (unsigned long long)total);
}

// Lanes per request for lookup: enough groups in flight to cover the chip
// (about 2^18 lanes), one lane each when the batch alone is that large; and,
// up to about 2^21 lanes, one lane per ~16 blocks of the average request,
// since a group walks its request's blocks G at a time and the longest
// request bounds the launch (a batch of long requests would otherwise wait on
// its longest one with one or two lanes).
//
// Batches of long requests (128 blocks or more on average) go to a full wave
// per request, up to 2^22 lanes: the launch then ends when the longest
// request's last round does, and a request of L blocks takes L / G rounds
// (65,536 requests averaging 208 blocks, at most 2048: 1.65 / 1.00 ms per
// lookup with 16 lanes per request, 1.34 / 0.75 ms with 64).  Short
// requests keep fewer lanes: their probes stop at the first miss, and spare
// lanes would only probe past it (1M probes of 8..64 blocks: 0.43 ms with 2
// lanes, 0.45 ms with 4).
static int lookup_group(int32_t n, int64_t n_blocks) {
  int g = 1;
  while (g < 64 && (int64_t)n * g * 2 <= (1 << 18)) g <<= 1;
  const int64_t avg = n > 0 ? n_blocks / n : 0;
  while (g < 64 && (int64_t)g * 16 <= avg && (int64_t)n * g * 2 <= (1 << 21)) g <<= 1;
  if (avg >= 128)
    while (g < 64 && (int64_t)n * g * 2 <= (1 << 22)) g <<= 1;
  return g;
}

}  // namespace kvgov

using namespace kvgov;

namespace {

int check_device(const kvgov_cache *c) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return KVGOV_E_HIP;
  return dev == c->device ? KVGOV_OK : KVGOV_E_DEVICE;
}

unsigned grid_for(int64_t work, int per_cu) {
  const int64_t cap = (int64_t)device_cu_count() * per_cu;
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(work, 256), cap));
}

// The recency words are rewritten only if something may have written them
// since they were last cleared (a tracked insert or admission, an eviction,
// an erasure): on a table that never tracks, a clear writes 40 of its 48
// bytes per slot.
int enqueue_clear(kvgov_cache *c, hipStream_t s) {
  hipLaunchKernelGGL(k_cache_fill, dim3(grid_for(c->slots, 64)), dim3(256), 0, s, c->view.keys,
                     c->view.tags, c->rank_dirty ? c->view.rank : nullptr, c->slots,
                     c->view.meta);
  c->rank_dirty = false;
  c->epoch.store(0);
  return launch_status();
}

// The plain insert takes a group of lanes per request while requests
// average at most this many rows (a group walks its request 64 rows at a
// time, so one request of 2^20 rows would take 16k steps of one wave), and
// the chunked walk above it.
constexpr int64_t kReqInsertMaxAvg = 4096;

// Lanes per request of the plain insert: about one lane per two rows of
// the average request, 4 to 64.
int insert_group(int32_t n, int64_t n_blocks) {
  const int64_t avg = n > 0 ? n_blocks / n : 0;
  int g = 4;
  while (g < 64 && (int64_t)g * 2 < avg) g <<= 1;
  return g;
}

// k_chunk_insert: waves of 4 x kInsChunk keys, at most 16 workgroups per CU.
unsigned insert_grid(int64_t n_blocks) {
  const int64_t groups = ceil_div(std::max<int64_t>(n_blocks, 1), (int64_t)kInsChunk * 4);
  return (unsigned)std::min<int64_t>(groups, (int64_t)device_cu_count() * 16);
}

int read_meta(kvgov_cache *c, CacheMeta *m, hipStream_t s) {
  if (hipMemcpyAsync(m, c->view.meta, sizeof(CacheMeta), hipMemcpyDeviceToHost, s) !=
      hipSuccess)
    return KVGOV_E_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return KVGOV_E_HIP;
  return KVGOV_OK;
}

// Maintenance scratch, in the stream's scratch buffer: selection state, the
// rank histogram and room for every key of the table (32 B key + 8 B recency
// each).  `lk` holds the scratch registry while the call enqueues its
// kernels; the stream runs its calls in order, so the buffer serves this
// call until its kernels end.
struct MaintScratch {
  SelectState *st = nullptr;
  unsigned int *hist = nullptr;
  u32x4 *keys = nullptr;
  unsigned long long *rank = nullptr;
  int64_t cap = 0;
  std::unique_lock<std::mutex> lk;
};

// Workgroups of the compaction kernels: one step of 4096 slots each, at most
// 4 per CU.
unsigned compact_grid(int64_t slots) {
  return (unsigned)std::max<int64_t>(
      1, std::min<int64_t>(ceil_div(slots, 256 * kCompactItems), (int64_t)device_cu_count() * 4));
}

int maint_alloc(kvgov_cache *c, hipStream_t s, MaintScratch &m) {
  m.cap = c->slots + 1;
  const size_t off_hist = 256;
  const size_t off_keys = off_hist + kRankBins * sizeof(unsigned int);
  const size_t off_rank = off_keys + (size_t)m.cap * 32;
  const size_t bytes = off_rank + (size_t)m.cap * 8;
  void *base = nullptr;
  const int rc = stream_scratch(s, bytes, &base, m.lk);
  if (rc != KVGOV_OK) return rc;
  uint8_t *b = static_cast<uint8_t *>(base);
  m.st = reinterpret_cast<SelectState *>(b);
  m.hist = reinterpret_cast<unsigned int *>(b + off_hist);
  m.keys = reinterpret_cast<u32x4 *>(b + off_keys);
  m.rank = reinterpret_cast<unsigned long long *>(b + off_rank);
  return KVGOV_OK;
}

// Copies out what ranks at or above the selected threshold, empties the
// table and inserts the copies again; then reads one counter if asked
// (waiting for the stream).
int compact_rebuild(kvgov_cache *c, hipStream_t s, MaintScratch &m, const unsigned long long *count,
                    int64_t *out) {
  const uint32_t epoch = c->epoch.fetch_add(1) + 1;
  int rc = epoch == 0xFFFFFFFFu ? KVGOV_E_UNSUPPORTED : KVGOV_OK;
  if (rc == KVGOV_OK) {
    hipLaunchKernelGGL(k_compact, dim3(compact_grid(c->slots)), dim3(256), 0, s, c->view, m.st,
                       m.keys, m.rank, m.cap);
    hipLaunchKernelGGL(k_rebuild_fill, dim3(grid_for(c->slots, 64)), dim3(256), 0, s, c->view);
    hipLaunchKernelGGL(k_reinsert, dim3(grid_for(m.cap, 16)), dim3(256), 0, s, c->view, m.st,
                       reinterpret_cast<const uint8_t *>(m.keys), m.rank, epoch, m.cap);
    rc = launch_status();
  }
  unsigned long long host = 0;
  if (rc == KVGOV_OK && out &&
      hipMemcpyAsync(&host, count, sizeof host, hipMemcpyDeviceToHost, s) != hipSuccess)
    rc = KVGOV_E_HIP;
  if (m.lk.owns_lock()) m.lk.unlock();  // everything that uses the scratch is enqueued
  if (rc == KVGOV_OK && out) {
    if (hipStreamSynchronize(s) != hipSuccess) return KVGOV_E_HIP;
    *out = (int64_t)host;
    CacheMeta meta{};
    rc = read_meta(c, &meta, s);
    if (rc == KVGOV_OK) rc = meta.status;
  }
  return rc;
}

// Keys added by insert call `epoch` (waits for the stream), and the latched
// error.
int read_new_keys(kvgov_cache *c, uint32_t epoch, int64_t *n_new, hipStream_t s) {
  CacheMeta m{};
  int rc = read_meta(c, &m, s);
  if (rc != KVGOV_OK) return rc;
  int64_t added = 0;
  for (int i = 0; i < kCounterLanes; ++i) added += (int64_t)m.new_keys[epoch & 1][i];
  *n_new = added;
  return m.status;
}

}  // namespace

int kvgov::cache_insert_rows(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                             int32_t n, int64_t n_blocks, hipStream_t s, uint32_t *epoch) {
  *epoch = c->epoch.fetch_add(1) + 1;
  if (*epoch == 0xFFFFFFFFu) return KVGOV_E_UNSUPPORTED;  // 2^32 - 1 inserts since clear
  if (c->view.track) c->rank_dirty = true;
  if (n == 0) {
    // no request: only the batch check and the next call's counters
    hipLaunchKernelGGL(k_insert_req<64>, dim3(1), dim3(256), 0, s, c->view, hashes, blk_offsets,
                       n, n_blocks, *epoch);
    return launch_status();
  }
  if (n_blocks > (int64_t)n * kReqInsertMaxAvg) {
    // few, long requests: a group per request would leave the chip idle
    hipLaunchKernelGGL(k_chunk_insert<false>, dim3(insert_grid(n_blocks)), dim3(256), 0, s,
                       c->view, hashes, blk_offsets, n, n_blocks, *epoch, nullptr);
    return launch_status();
  }
  const int g = insert_group(n, n_blocks);
  const dim3 grid((unsigned)ceil_div((int64_t)n * g, 256)), block(256);
  switch (g) {
    case 4: hipLaunchKernelGGL(k_insert_req<4>, grid, block, 0, s, c->view, hashes, blk_offsets, n, n_blocks, *epoch); break;
    case 8: hipLaunchKernelGGL(k_insert_req<8>, grid, block, 0, s, c->view, hashes, blk_offsets, n, n_blocks, *epoch); break;
    case 16: hipLaunchKernelGGL(k_insert_req<16>, grid, block, 0, s, c->view, hashes, blk_offsets, n, n_blocks, *epoch); break;
    case 32: hipLaunchKernelGGL(k_insert_req<32>, grid, block, 0, s, c->view, hashes, blk_offsets, n, n_blocks, *epoch); break;
    default: hipLaunchKernelGGL(k_insert_req<64>, grid, block, 0, s, c->view, hashes, blk_offsets, n, n_blocks, *epoch); break;
  }
  return launch_status();
}

extern "C" {

int kvgov_cache_create(int32_t log2_slots, kvgov_cache **out) {
  if (!out || log2_slots < KVGOV_MIN_LOG2_SLOTS || log2_slots > KVGOV_MAX_LOG2_SLOTS)
    return KVGOV_E_INVAL;
  *out = nullptr;
  kvgov_cache *c = new (std::nothrow) kvgov_cache();
  if (!c) return KVGOV_E_NOMEM;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return KVGOV_E_HIP;
  }
  c->log2_slots = log2_slots;
  c->slots = (int64_t)1 << log2_slots;
  c->view.mask = (uint64_t)c->slots - 1;
  void *keys = nullptr, *tags = nullptr, *rank = nullptr, *meta = nullptr;
  if (hipMalloc(&keys, (size_t)c->slots * 32) != hipSuccess ||
      hipMalloc(&tags, (size_t)c->slots * 8) != hipSuccess ||
      hipMalloc(&rank, (size_t)c->slots * 8) != hipSuccess ||
      hipMalloc(&meta, sizeof(CacheMeta)) != hipSuccess) {
    if (keys) (void)hipFree(keys);
    if (tags) (void)hipFree(tags);
    if (rank) (void)hipFree(rank);
    if (meta) (void)hipFree(meta);
    delete c;
    return KVGOV_E_NOMEM;
  }
  c->view.keys = static_cast<u32x4 *>(keys);
  c->view.tags = static_cast<unsigned long long *>(tags);
  c->view.rank = static_cast<unsigned long long *>(rank);
  c->view.track = 0;
  c->view.meta = static_cast<CacheMeta *>(meta);
  int rc = enqueue_clear(c, nullptr);
  if (rc == KVGOV_OK && hipStreamSynchronize(nullptr) != hipSuccess) rc = KVGOV_E_HIP;
  if (rc != KVGOV_OK) {
    kvgov_cache_destroy(c);
    return rc;
  }
  *out = c;
  return KVGOV_OK;
}

int kvgov_cache_destroy(kvgov_cache *c) {
  if (!c) return KVGOV_OK;
  int rc = KVGOV_OK;
  if (hipDeviceSynchronize() != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(c->view.keys) != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(c->view.tags) != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(c->view.rank) != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(c->view.meta) != hipSuccess) rc = KVGOV_E_HIP;
  delete c;
  return rc;
}

int kvgov_cache_clear(kvgov_cache *c, void *stream) {
  if (!c) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  return enqueue_clear(c, as_stream(stream));
}

int kvgov_cache_slots(const kvgov_cache *c, int64_t *slots) {
  if (!c || !slots) return KVGOV_E_INVAL;
  *slots = c->slots;
  return KVGOV_OK;
}

int kvgov_cache_insert(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                       int32_t n, int64_t n_blocks, int64_t *n_new, void *stream) {
  if (!c || !blk_offsets || n < 0 || n_blocks < 0 || (n_blocks > 0 && !hashes))
    return KVGOV_E_INVAL;
  if (reinterpret_cast<uintptr_t>(hashes) & 3) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  hipStream_t s = as_stream(stream);
  uint32_t epoch = 0;
  rc = cache_insert_rows(c, hashes, blk_offsets, n, n_blocks, s, &epoch);
  if (rc != KVGOV_OK || !n_new) return rc;
  return read_new_keys(c, epoch, n_new, s);
}

int kvgov_cache_lookup(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                       int32_t n, int64_t n_blocks, int32_t *hit_blocks, void *stream) {
  if (!c || !blk_offsets || n < 0 || n_blocks < 0 || (n_blocks > 0 && !hashes) ||
      (n > 0 && !hit_blocks))
    return KVGOV_E_INVAL;
  if (reinterpret_cast<uintptr_t>(hashes) & 3) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  if (n == 0) return KVGOV_OK;
  hipStream_t s = as_stream(stream);
  LookupArgs a{c->view, hashes, blk_offsets, n, n_blocks, hit_blocks};
  const int g = lookup_group(n, n_blocks);
  const dim3 grid((unsigned)ceil_div((int64_t)n * g, 256)), block(256);
  switch (g) {
    case 1: hipLaunchKernelGGL(k_lookup<1>, grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL(k_lookup<2>, grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL(k_lookup<4>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(k_lookup<8>, grid, block, 0, s, a); break;
    case 16: hipLaunchKernelGGL(k_lookup<16>, grid, block, 0, s, a); break;
    case 32: hipLaunchKernelGGL(k_lookup<32>, grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL(k_lookup<64>, grid, block, 0, s, a); break;
  }
  return launch_status();
}

// Lanes per request for the admission scan, which walks every row of a
// request: about one lane per 2 rows of the average request, 4 to 64.
static int admit_group(int32_t n, int64_t n_blocks) {
  const int64_t avg = n > 0 ? n_blocks / n : 0;
  int g = 4;
  while (g < 64 && (int64_t)g * 2 < avg) g <<= 1;
  return g;
}

int kvgov_cache_admit(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                      int32_t n, int64_t n_blocks, int32_t *hit_blocks, int32_t *new_blocks,
                      int64_t *n_new, void *stream) {
  if (!c || !blk_offsets || n < 0 || n_blocks < 0 || (n_blocks > 0 && !hashes) ||
      (n > 0 && (!hit_blocks || !new_blocks)))
    return KVGOV_E_INVAL;
  if (reinterpret_cast<uintptr_t>(hashes) & 3) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  if (n == 0) {
    if (n_new) *n_new = 0;
    return KVGOV_OK;
  }
  hipStream_t s = as_stream(stream);
  // per-row codes of the insert, in the stream's scratch (held while the two
  // kernels are enqueued)
  std::unique_lock<std::mutex> lk;
  void *scratch_p = nullptr;
  rc = stream_scratch(s, sizeof(uint32_t) * (size_t)std::max<int64_t>(n_blocks, 1), &scratch_p,
                      lk);
  if (rc != KVGOV_OK) return rc;
  uint32_t *codes = static_cast<uint32_t *>(scratch_p);
  const uint32_t epoch = c->epoch.fetch_add(1) + 1;
  if (epoch == 0xFFFFFFFFu) return KVGOV_E_UNSUPPORTED;
  if (c->view.track) c->rank_dirty = true;
  hipLaunchKernelGGL(k_chunk_insert<true>, dim3(insert_grid(n_blocks)), dim3(256), 0, s,
                     c->view, hashes, blk_offsets, n, n_blocks, epoch, codes);
  AdmitArgs a{c->view, blk_offsets, n, n_blocks, epoch, codes, hit_blocks, new_blocks};
  const int g = admit_group(n, n_blocks);
  const dim3 grid((unsigned)ceil_div((int64_t)n * g, 256)), block(256);
  switch (g) {
    case 4: hipLaunchKernelGGL(k_admit_scan<4>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(k_admit_scan<8>, grid, block, 0, s, a); break;
    case 16: hipLaunchKernelGGL(k_admit_scan<16>, grid, block, 0, s, a); break;
    case 32: hipLaunchKernelGGL(k_admit_scan<32>, grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL(k_admit_scan<64>, grid, block, 0, s, a); break;
  }
  rc = launch_status();
  lk.unlock();
  if (rc != KVGOV_OK || !n_new) return rc;
  return read_new_keys(c, epoch, n_new, s);
}

int kvgov_cache_set_recency(kvgov_cache *c, int32_t on) {
  if (!c || (on != 0 && on != 1)) return KVGOV_E_INVAL;
  c->view.track = (uint32_t)on;
  return KVGOV_OK;
}

int kvgov_cache_evict(kvgov_cache *c, int64_t max_keys, int64_t *n_kept, void *stream) {
  if (!c || max_keys < 0) return KVGOV_E_INVAL;
  if (!c->view.track) return KVGOV_E_UNSUPPORTED;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  hipStream_t s = as_stream(stream);
  MaintScratch m;
  rc = maint_alloc(c, s, m);
  if (rc != KVGOV_OK) return rc;
  hipLaunchKernelGGL(k_select_init, dim3(1), dim3(kRankBins), 0, s, m.st, m.hist,
                     (long long)max_keys, 0);
  // the gathered words live in the key area of the scratch until the
  // compaction overwrites it
  unsigned long long *dense = reinterpret_cast<unsigned long long *>(m.keys);
  hipLaunchKernelGGL(k_gather_ranks, dim3(compact_grid(c->slots)), dim3(256), 0, s, c->view,
                     m.st, dense);
  hipLaunchKernelGGL(k_select_start, dim3(1), dim3(1), 0, s, m.st);
  for (int level = 0; level < 8; ++level) {
    hipLaunchKernelGGL(k_rank_hist, dim3(grid_for(c->slots, 4)), dim3(256), 0, s, m.st, dense,
                       m.hist);
    hipLaunchKernelGGL(k_rank_select, dim3(1), dim3(kRankBins), 0, s, m.st, m.hist);
  }
  c->rank_dirty = true;
  return compact_rebuild(c, s, m, &m.st->kept, n_kept);
}

int kvgov_cache_erase(kvgov_cache *c, const uint8_t *keys, int64_t n_keys, int64_t *n_erased,
                      void *stream) {
  if (!c || n_keys < 0 || (n_keys > 0 && !keys)) return KVGOV_E_INVAL;
  if (reinterpret_cast<uintptr_t>(keys) & 3) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  hipStream_t s = as_stream(stream);
  MaintScratch m;
  rc = maint_alloc(c, s, m);
  if (rc != KVGOV_OK) return rc;
  hipLaunchKernelGGL(k_select_init, dim3(1), dim3(kRankBins), 0, s, m.st, m.hist, 0ll, 1);
  if (n_keys > 0)
    hipLaunchKernelGGL(k_erase_mark, dim3((unsigned)ceil_div(n_keys, 256)), dim3(256), 0, s,
                       c->view, keys, n_keys, m.st);
  c->rank_dirty = true;
  return compact_rebuild(c, s, m, &m.st->erased, n_erased);
}

int kvgov_cache_count(kvgov_cache *c, int64_t *n_keys, void *stream) {
  if (!c || !n_keys) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  CacheMeta m{};
  rc = read_meta(c, &m, as_stream(stream));
  if (rc != KVGOV_OK) return rc;
  int64_t total = 0;
  for (int i = 0; i < kCounterLanes; ++i) total += (int64_t)m.n_keys[i];
  *n_keys = total;
  return m.status;
}

int kvgov_cache_export(kvgov_cache *c, uint8_t *keys, int64_t cap, int64_t *n_keys,
                       void *stream) {
  if (!c || !n_keys || cap < 0 || (cap > 0 && !keys)) return KVGOV_E_INVAL;
  if (reinterpret_cast<uintptr_t>(keys) & 3) return KVGOV_E_INVAL;
  int rc = check_device(c);
  if (rc != KVGOV_OK) return rc;
  hipStream_t s = as_stream(stream);
  hipLaunchKernelGGL(k_export_begin, dim3(1), dim3(1), 0, s, c->view.meta);
  hipLaunchKernelGGL(k_export, dim3(grid_for(c->slots, 32)), dim3(256), 0, s, c->view, keys,
                     cap);
  rc = launch_status();
  if (rc != KVGOV_OK) return rc;
  CacheMeta m{};
  rc = read_meta(c, &m, s);
  if (rc != KVGOV_OK) return rc;
  *n_keys = (int64_t)m.exported;
  return (int64_t)m.exported > cap ? KVGOV_E_CAPACITY : KVGOV_OK;
}

}  // extern "C"
