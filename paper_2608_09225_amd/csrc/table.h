// Device-resident hash table of 32-byte keys shared by the prefix cache
// (cache.hip) and the radix index (radix.hip): layout, key helpers, the
// insert protocol and probes.  Internal to libkvgov.
#pragma once

#include <atomic>

#include "common.h"

namespace kvgov {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4), aligned(4)));

// Counters are spread over kCounterLanes addresses (a workgroup adds to lane
// blockIdx % kCounterLanes): atomics on one address serialise at ~10 ns each,
// which at one atomic per wave dominated a 680k-key insert.  Readers sum.
constexpr int kCounterLanes = 64;

struct CacheMeta {
  unsigned long long n_keys[kCounterLanes];       // keys in the table (all-0xFF key included)
  unsigned long long new_keys[2][kCounterLanes];  // keys added by insert call `epoch`, at [epoch & 1]
  unsigned long long exported;                    // keys written by the latest export
  unsigned long long ones_tag;                    // the all-0xFF key's tag (0 = absent)
  unsigned long long ones_rank;                   // its recency rank (as `rank`)
  int32_t status;                                 // latched error (0 = none)
  int32_t ones_present;                           // the all-0xFF key is in the table
};

// Recency of a key (table maintenance, when the table tracks it): one word,
// (stamp << 32) | (kNoDepth - depth), where the stamp is the epoch of the
// latest insert or admission call whose batch held the key and the depth
// the smallest row position (within its request) the key had in that call.
// Newer calls rank higher, and within a call shallower positions; both are
// raised by one atomicMax.  0 = never touched; kErased marks a key an erase
// call is removing.
constexpr uint32_t kNoDepth = 0xFFFFFFFFu;
constexpr unsigned long long kErased = ~0ull;

struct TableView {
  u32x4 *keys;  // 2 per slot
  unsigned long long *tags;
  unsigned long long *rank;  // recency word per slot
  CacheMeta *meta;
  uint64_t mask;   // slots - 1
  uint32_t track;  // inserts and admissions raise `rank`
};

struct Key {
  u32x4 lo, hi;
};

__device__ __forceinline__ Key load_key(const uint8_t *p) {
  const u32x4 *q = reinterpret_cast<const u32x4 *>(p);
  return Key{q[0], q[1]};
}

__device__ __forceinline__ bool key_eq(const Key &a, const Key &b) {
  const uint32_t d = (a.lo.x ^ b.lo.x) | (a.lo.y ^ b.lo.y) | (a.lo.z ^ b.lo.z) |
                     (a.lo.w ^ b.lo.w) | (a.hi.x ^ b.hi.x) | (a.hi.y ^ b.hi.y) |
                     (a.hi.z ^ b.hi.z) | (a.hi.w ^ b.hi.w);
  return d == 0;
}

__device__ __forceinline__ bool key_is_empty_pattern(const Key &a) {
  return (a.lo.x & a.lo.y & a.lo.z & a.lo.w & a.hi.x & a.hi.y & a.hi.z & a.hi.w) ==
         0xFFFFFFFFu;
}

// Slot index from all 256 bits (keys are digests, but any 32-byte value is
// valid, so every word takes part), finished with a 64-bit mixer.
__device__ __forceinline__ uint64_t slot_hash(const Key &k) {
  uint64_t x = ((uint64_t)k.lo.y << 32 | k.lo.x) ^
               (((uint64_t)k.lo.w << 32 | k.lo.z) * 0x9E3779B97F4A7C15ull) ^
               (((uint64_t)k.hi.y << 32 | k.hi.x) * 0xC2B2AE3D27D4EB4Full) ^
               (((uint64_t)k.hi.w << 32 | k.hi.z) * 0x165667B19E3779F9ull);
  x ^= x >> 31;
  x *= 0xBF58476D1CE4E5B9ull;
  x ^= x >> 29;
  return x;
}

// A key's probe sequence starts at its home slot, runs through the rest of
// the home slot's bucket (four slots: one 128-byte line of keys), wrapping
// inside it, and then through the following buckets in the same way.  A
// search that runs past its home slot mostly finds the key, or an empty
// slot, in the line it has already read; plain linear probing crossed into
// the next line whenever a run reached the end of one (probe-heavy lookup:
// 2.40 -> 2.27 GB fetched, 0.432 -> 0.425 ms).  Measured alternatives, not
// used: probe sequences starting at the bucket's first slot made the
// insert of 13.7M distinct keys 15-20 % slower (a key's first slot is then
// four times as often claimed by another key of the same call, whose input
// row the insert reads to compare); reading a whole bucket with one lane
// (eight 16-byte loads per probe) made the lookup 9 % slower.
__device__ __forceinline__ uint64_t home_slot(const Key &k, uint64_t mask) {
  return slot_hash(k) & mask;
}

// probe p of the sequence from `home`: the four slots of home's bucket (one
// 128-byte line of keys) starting at home, then the next bucket's from the
// same offset, and so on
__device__ __forceinline__ uint64_t seq_slot(uint64_t home, uint64_t p, uint64_t mask) {
  return ((((home >> 2) + (p >> 2)) << 2) & mask) | ((home + p) & 3);
}

// Sum of v over the workgroup (256 threads), valid in thread 0.
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t *lds4) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  if ((threadIdx.x & 63) == 0) lds4[threadIdx.x >> 6] = v;
  __syncthreads();
  return threadIdx.x == 0 ? lds4[0] + lds4[1] + lds4[2] + lds4[3] : 0;
}

// Per-row codes written by the admission insert: the slot of the row's key,
// or one of these (slots < 2^31, so no slot index collides with them).
constexpr uint32_t kCodeOnes = 0xFFFFFFFEu;    // the all-0xFF key (tag in meta)
constexpr uint32_t kCodeDup = 0xFFFFFFFDu;     // equals the previous request's key here
constexpr uint32_t kCodeFailed = 0xFFFFFFFCu;  // not inserted (table full)

// A tag claimed in this call (same epoch) whose row is above `mine`: lower
// it.  Reads first, so most copies of a hot key issue no atomic.
__device__ __forceinline__ void lower_claim(unsigned long long *tag, unsigned long long seen,
                                            unsigned long long mine) {
  if (mine < seen) atomicMin(tag, mine);
}

// Raises a key's recency word to `mine`.  The word only grows within a
// call, so a plain read (possibly a stale line of this XCD's L2) that already
// shows `mine` or more ends it; otherwise a device-coherent read, and an
// atomic only where it changes something: a hot key held by thousands of
// rows costs a few atomics.  The row that just claimed the slot goes
// straight to the atomic.
__device__ __forceinline__ void touch(unsigned long long *w, unsigned long long mine,
                                      bool claimed) {
  if (!claimed) {
    if (*w >= mine) return;
    if (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= mine) return;
  }
  atomicMax(w, mine);
}

__device__ __forceinline__ unsigned long long recency(uint32_t epoch, uint32_t depth) {
  return ((unsigned long long)epoch << 32) | (unsigned long long)(kNoDepth - depth);
}

// Tags only ever change from 0 to a claim (and, within the claiming call, to
// a smaller claim of the same key), so a plain (possibly stale) read can only
// show 0 for a claimed slot; the compare-and-swap that follows then fails
// and returns the claim.  Coherent atomics are used for the claim only.
// Returns 1 if the key was added; *code receives where the key went, and
// *claim (if given) the key's tag as this lane found it (its own claim if it
// added the key).  On a table that tracks recency the key (added or found)
// is touched with (epoch, depth) unless depth is kNoDepth.
template <bool ADMIT>
__device__ __forceinline__ uint32_t insert_key(const TableView &t, const Key &key, int64_t i,
                                               int64_t lo, const uint8_t *hashes,
                                               uint32_t epoch, uint32_t *code,
                                               uint32_t depth = kNoDepth,
                                               unsigned long long *claim = nullptr) {
  const unsigned long long mine = ((unsigned long long)epoch << 32) |
                                  (unsigned long long)(i - lo + 1);
  if (key_is_empty_pattern(key)) {
    *code = kCodeOnes;
    unsigned long long expect = 0;
    const bool won = __hip_atomic_compare_exchange_strong(
        &t.meta->ones_tag, &expect, mine, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
        __HIP_MEMORY_SCOPE_AGENT);
    if (claim) *claim = won ? mine : expect;
    if (won) atomicExch(&t.meta->ones_present, 1);
    if (!won && ADMIT && (uint32_t)(expect >> 32) == epoch)
      lower_claim(&t.meta->ones_tag, expect, mine);
    if (t.track && depth != kNoDepth) touch(&t.meta->ones_rank, recency(epoch, depth), won);
    return won ? 1u : 0u;
  }
  const uint64_t home = home_slot(key, t.mask);
  for (uint64_t probes = 0; probes <= t.mask; ++probes) {
    const uint64_t s = seq_slot(home, probes, t.mask);
    unsigned long long tag = t.tags[s];
    if (tag == 0) {
      unsigned long long expect = 0;
      if (__hip_atomic_compare_exchange_strong(&t.tags[s], &expect, mine, __ATOMIC_RELAXED,
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        t.keys[2 * s] = key.lo;
        t.keys[2 * s + 1] = key.hi;
        *code = (uint32_t)s;
        if (claim) *claim = mine;
        if (t.track && depth != kNoDepth) touch(&t.rank[s], recency(epoch, depth), true);
        return 1;
      }
      tag = expect;  // somebody claimed it first: examine the claimant
    }
    Key other;
    const bool current = (uint32_t)(tag >> 32) == epoch;
    if (current) {
      const int64_t c = (int64_t)(tag & 0xFFFFFFFFull) - 1;
      other = load_key(hashes + (lo + c) * 32);
    } else {
      other = Key{t.keys[2 * s], t.keys[2 * s + 1]};
    }
    if (key_eq(key, other)) {
      if (ADMIT && current) lower_claim(&t.tags[s], tag, mine);
      *code = (uint32_t)s;
      if (claim) *claim = tag;
      if (t.track && depth != kNoDepth) touch(&t.rank[s], recency(epoch, depth), false);
      return 0;
    }
  }
  atomicCAS(&t.meta->status, 0, KVGOV_E_FULL);
  *code = kCodeFailed;
  if (claim) *claim = 0;
  return 0;
}

// Is `key` in the table?  Reads the key array only, one slot at a time (the
// slots after the first are mostly in its line, so their loads hit the cache).
__device__ __forceinline__ bool probe(const TableView &t, const Key &key, bool ones_present) {
  if (key_is_empty_pattern(key)) return ones_present;
  const uint64_t home = home_slot(key, t.mask);
  for (uint64_t p = 0; p <= t.mask; ++p) {
    const uint64_t s = seq_slot(home, p, t.mask);
    const Key slot{t.keys[2 * s], t.keys[2 * s + 1]};
    if (key_eq(slot, key)) return true;
    if (key_is_empty_pattern(slot)) return false;
  }
  return false;
}

// Lanes of a G-lane group starting at lane `base` of the wave.
template <int G>
__device__ __forceinline__ uint64_t group_mask(int base) {
  if constexpr (G == 64) {
    return ~0ull;
  } else {
    return ((1ull << G) - 1ull) << base;
  }
}

// Slot holding `key`, or -1 (the all-0xFF key has no slot: -2 if present).
__device__ __forceinline__ int64_t find_slot(const TableView &t, const Key &key) {
  if (key_is_empty_pattern(key)) return t.meta->ones_present ? -2 : -1;
  const uint64_t home = home_slot(key, t.mask);
  for (uint64_t p = 0; p <= t.mask; ++p) {
    const uint64_t s = seq_slot(home, p, t.mask);
    const Key slot{t.keys[2 * s], t.keys[2 * s + 1]};
    if (key_eq(slot, key)) return (int64_t)s;
    if (key_is_empty_pattern(slot)) return -1;
  }
  return -1;
}

// Enqueues the plain set-union insert of a batch's rows (cache.hip); stores
// the call's epoch, whose tags mark the slots the call claimed, each with
// the row that claimed it.
int cache_insert_rows(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                      int32_t n, int64_t n_blocks, hipStream_t s, uint32_t *epoch);

}  // namespace kvgov

// The table object behind kvgov_cache *.
struct kvgov_cache {
  int device;
  int32_t log2_slots;
  int64_t slots;
  kvgov::TableView view;  // view.track: recency tracking on
  std::atomic<uint32_t> epoch;
  // recency words may be nonzero (set when a call that can write them is
  // enqueued; the next clear rewrites them)
  std::atomic<bool> rank_dirty{true};
};

