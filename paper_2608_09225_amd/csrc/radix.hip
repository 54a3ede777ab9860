// Token-granular prefix index: the radix-tree row of the paper's cache
// taxonomy (Table tab:taxonomy; Sec. 3.5: a radix tree reports the matched
// prefix length in tokens, finer than whole blocks), with the per-principal
// root of Sec. 4.1 (sigma_p as the root node gives each principal a disjoint
// tree).
//
// Structure: a trie whose nodes are
//   * block nodes: the chained digest h_j of a full block (the same keys as
//     the block prefix cache) and the roots (sigma_p, or 32 zero bytes for
//     the unsalted tree), stored in a block table (table.h); a node's id is
//     its slot index;
//   * token nodes: the prefixes of 1..15 tokens of a block below its parent
//     block node, stored as edges (parent id, token) -> child in an edge table
//     of 64-bit keys; a child's id is kEdgeBase + its edge slot.
// A full block leads from the node of h_{j-1} to the node of h_j (through the
// block table: the 16th token is never an edge); a partial last block of an
// inserted sequence ends at a token node.  Match: the first block whose digest
// is absent gives the block depth m, and the longest walk of edges from the
// node of h_{m-1} over the request's next tokens (at most 15) gives the rest:
// match = 16 m + steps.  The 16th step cannot exist: it would make block m
// present.
//
// Edge insert is one 64-bit compare-and-swap per edge (the key is the whole
// slot), so no lane ever reads a slot another lane is still writing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <new>

#include "table.h"

namespace kvgov {

constexpr unsigned long long kEdgeEmpty = ~0ull;
constexpr uint32_t kEdgeBase = 0x80000000u;  // id of the token node in edge slot e
constexpr uint32_t kOnesNode = 0x7FFFFFFFu;  // id of the all-0xFF block key (no slot)
constexpr uint32_t kNoNode = 0xFFFFFFFFu;
constexpr int kMaxLog2Radix = 30;           // keeps slot ids clear of the ids above

struct RadixMeta {
  unsigned long long n_edges[kCounterLanes];
  int32_t status;
};

struct EdgeView {
  unsigned long long *keys;
  uint64_t mask;
  RadixMeta *meta;
};

__device__ __forceinline__ uint64_t edge_hash(unsigned long long k) {
  uint64_t x = k * 0x9E3779B97F4A7C15ull;
  x ^= x >> 32;
  x *= 0xD6E8FEB86659FD93ull;
  x ^= x >> 32;
  return x;
}

__device__ __forceinline__ unsigned long long edge_key(uint32_t node, int32_t tok) {
  return ((unsigned long long)node << 32) | (uint32_t)tok;
}

// Child id of edge (node, tok), creating it if absent; kNoNode if the table
// is full (latched).  *added counts a created edge.
__device__ __forceinline__ uint32_t edge_insert(const EdgeView &e, uint32_t node, int32_t tok,
                                                uint32_t *added) {
  const unsigned long long key = edge_key(node, tok);
  uint64_t s = edge_hash(key) & e.mask;
  for (uint64_t p = 0; p <= e.mask; ++p) {
    unsigned long long cur = e.keys[s];
    if (cur == kEdgeEmpty) {
      cur = atomicCAS(&e.keys[s], kEdgeEmpty, key);
      if (cur == kEdgeEmpty) {
        ++*added;
        return kEdgeBase + (uint32_t)s;
      }
    }
    if (cur == key) return kEdgeBase + (uint32_t)s;
    s = (s + 1) & e.mask;
  }
  atomicCAS(&e.meta->status, 0, KVGOV_E_FULL);
  return kNoNode;
}

__device__ __forceinline__ uint32_t edge_find(const EdgeView &e, uint32_t node, int32_t tok) {
  const unsigned long long key = edge_key(node, tok);
  uint64_t s = edge_hash(key) & e.mask;
  for (uint64_t p = 0; p <= e.mask; ++p) {
    const unsigned long long cur = e.keys[s];
    if (cur == key) return kEdgeBase + (uint32_t)s;
    if (cur == kEdgeEmpty) return kNoNode;
    s = (s + 1) & e.mask;
  }
  return kNoNode;
}

// Node id of a block key (kNoNode if absent).
__device__ __forceinline__ uint32_t block_node(const TableView &t, const Key &k) {
  const int64_t s = find_slot(t, k);
  return s >= 0 ? (uint32_t)s : (s == -2 ? kOnesNode : kNoNode);
}

__global__ __launch_bounds__(256) void k_edge_fill(unsigned long long *keys, int64_t slots,
                                                   RadixMeta *m) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < kCounterLanes; i += blockDim.x) m->n_edges[i] = 0;
    if (threadIdx.x == 0) m->status = 0;
  }
  for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < slots; s += stride)
    keys[s] = kEdgeEmpty;
}

// Root keys into the block table (a row each; the insert protocol of
// table.h with `keys` as the call's input array).
__global__ __launch_bounds__(256) void k_radix_roots(TableView t, const uint8_t *keys,
                                                     int64_t count, uint32_t epoch) {
  uint32_t added = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * 256) {
    uint32_t code;
    added += insert_key<false>(t, load_key(keys + i * 32), i, 0, keys, epoch, &code, 0u);
  }
  if (added) atomicAdd(&t.meta->n_keys[blockIdx.x % kCounterLanes], (unsigned long long)added);
}

struct RadixArgs {
  TableView t;
  EdgeView e;
  const int32_t *tokens;
  int64_t n_tokens;
  const int64_t *tok_offsets;
  int32_t n;
  const int32_t *principal;
  const uint8_t *salts;  // ROOT: the roots; NONE: NULL (the zero root below)
  int32_t P;
  const uint8_t *zero_root;
  const uint8_t *hashes;
  const int64_t *blk_offsets;
  int64_t n_blocks;
  int32_t *match_len;  // match only
  uint32_t blk_epoch;  // insert only: the epoch of the call's block insert
};

// Request r's token range, full-block rows and root key, or false (latched).
struct RadixReq {
  int64_t t0, len, b0, nf;
  const uint8_t *root;
};

__device__ __forceinline__ bool radix_req(const RadixArgs &a, int64_t r, RadixReq &q) {
  q.t0 = a.tok_offsets[r];
  const int64_t t1 = a.tok_offsets[r + 1];
  q.b0 = a.blk_offsets[r];
  const int64_t b1 = a.blk_offsets[r + 1];
  q.len = t1 - q.t0;
  q.nf = b1 - q.b0;
  if (q.t0 < 0 || t1 < q.t0 || t1 > a.n_tokens || q.b0 < 0 || q.nf != (q.len >> 4) ||
      b1 > a.n_blocks) {
    atomicCAS(&a.e.meta->status, 0, KVGOV_E_OFFSETS);
    return false;
  }
  if (a.salts) {
    const int32_t p = a.principal[r];
    if (p < 0 || p >= a.P) {
      atomicCAS(&a.e.meta->status, 0, KVGOV_E_PRINCIPAL);
      return false;
    }
    q.root = a.salts + (int64_t)p * 32;
  } else {
    q.root = a.zero_root;
  }
  return true;
}

// Insert: G lanes per request, one (possibly partial) block each: the edges
// of its first min(len, 15) tokens below its parent block node.  The edges
// of a full block j are fixed by h_j (its parent and its tokens), so only
// the row that claimed h_j in this call's block insert walks them: a block
// present before the call has them already, and every other row holding
// h_j would repeat them (thousands of rows of a shared prefix would
// otherwise contend on the same edge slots).  A partial last block has no
// digest and always walks its edges.
template <int G>
__global__ __launch_bounds__(256) void k_radix_edges(RadixArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t r = gid / G;
  if (r >= a.n) return;
  const int sub = (int)(gid % G);
  RadixReq q;
  if (!radix_req(a, r, q)) return;
  uint32_t added = 0;
  const int64_t nrec = (q.len + 15) >> 4;  // full blocks and a partial tail
  const int64_t lo = a.blk_offsets[0];
  for (int64_t j = sub; j < nrec; j += G) {
    if (j < q.nf) {
      const int64_t f = q.b0 + j;
      const int64_t slot = find_slot(a.t, load_key(a.hashes + f * 32));
      if (slot >= 0) {
        const unsigned long long tag = a.t.tags[slot];
        if ((uint32_t)(tag >> 32) != a.blk_epoch ||
            (int64_t)(tag & 0xFFFFFFFFull) - 1 != f - lo)
          continue;  // not this row's block to expand
      }
      // slot < 0: the all-0xFF digest (no tag: expand, edges are idempotent)
      // or a block the full table could not take (the walk below latches)
    }
    uint32_t node = block_node(a.t, load_key(j == 0 ? q.root : a.hashes + (q.b0 + j - 1) * 32));
    if (node == kNoNode) {
      // the parent block was not inserted (a full table, latched there)
      atomicCAS(&a.e.meta->status, 0, KVGOV_E_FULL);
      continue;
    }
    const int64_t rem = q.len - 16 * j;
    const int steps = (int)(rem < 15 ? rem : 15);
    const int32_t *tp = a.tokens + q.t0 + 16 * j;
    for (int i = 0; i < steps && node != kNoNode; ++i) node = edge_insert(a.e, node, tp[i], &added);
  }
  if (added)
    atomicAdd(&a.e.meta->n_edges[blockIdx.x % kCounterLanes], (unsigned long long)added);
}

// Match: G lanes per request find the first absent block digest m (ballot),
// then one lane walks the edges below block node m - 1 (or the root).
template <int G>
__global__ __launch_bounds__(256) void k_radix_match(RadixArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t r = gid / G;
  if (r >= a.n) return;  // groups never straddle this test: 256 % G == 0
  const int sub = (int)(gid % G);
  const int lane = threadIdx.x & 63;
  const int base = lane & ~(G - 1);
  const uint64_t gmask = group_mask<G>(base);
  RadixReq q;
  if (!radix_req(a, r, q)) {
    if (sub == 0) a.match_len[r] = 0;
    return;
  }
  const bool ones = a.t.meta->ones_present != 0;
  int64_t m = q.nf;
  for (int64_t j0 = 0; j0 < q.nf; j0 += G) {
    const int64_t j = j0 + sub;
    bool miss = false;
    if (j < q.nf) miss = !probe(a.t, load_key(a.hashes + (q.b0 + j) * 32), ones);
    const uint64_t mk = __ballot(miss) & gmask;
    if (mk) {
      m = j0 + (__builtin_ctzll(mk) - base);
      break;
    }
  }
  if (sub != 0) return;
  uint32_t node = block_node(a.t, load_key(m == 0 ? q.root : a.hashes + (q.b0 + m - 1) * 32));
  int64_t steps = 0;
  if (node != kNoNode) {
    const int64_t rem = q.len - 16 * m;
    const int64_t lim = rem < 15 ? rem : 15;
    const int32_t *tp = a.tokens + q.t0 + 16 * m;
    while (steps < lim) {
      node = edge_find(a.e, node, tp[steps]);
      if (node == kNoNode) break;
      ++steps;
    }
  } else if (m > 0) {
    m = 0;  // cannot happen for a consistent table: h_{m-1} was just found
  }
  a.match_len[r] = (int32_t)(16 * m + steps);
}

}  // namespace kvgov

using namespace kvgov;

struct kvgov_radix {
  int device;
  kvgov_cache *blocks;
  EdgeView edges;
  int64_t edge_slots;
  uint8_t *zero_root;  // 32 zero bytes: the unsalted tree's root key
};

namespace {

int radix_check(const kvgov_radix *x) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return KVGOV_E_HIP;
  return dev == x->device ? KVGOV_OK : KVGOV_E_DEVICE;
}

int enqueue_edge_clear(kvgov_radix *x, hipStream_t s) {
  const unsigned grid = (unsigned)std::max<int64_t>(
      1, std::min<int64_t>(ceil_div(x->edge_slots, 256), (int64_t)device_cu_count() * 64));
  hipLaunchKernelGGL(k_edge_fill, dim3(grid), dim3(256), 0, s, x->edges.keys, x->edge_slots,
                     x->edges.meta);
  return launch_status();
}

// Lanes per request: about one per two blocks of the average request, 4..64.
int radix_group(int32_t n, int64_t n_blocks) {
  const int64_t avg = n > 0 ? n_blocks / n : 0;
  int g = 4;
  while (g < 64 && (int64_t)g * 2 < avg) g <<= 1;
  return g;
}

// Shared argument checks of insert and match; fills the kernel arguments.
int radix_args(kvgov_radix *x, const int32_t *tokens, int64_t n_tokens,
               const int64_t *tok_offsets, int32_t n, const int32_t *principal,
               const uint8_t *salts, int32_t P, int32_t mode, const uint8_t *hashes,
               const int64_t *blk_offsets, int64_t n_blocks, RadixArgs &a) {
  if (!x || n < 0 || n_tokens < 0 || n_blocks < 0) return KVGOV_E_INVAL;
  if (mode == KVGOV_BOUNDARY) return KVGOV_E_UNSUPPORTED;
  if (mode != KVGOV_NONE && mode != KVGOV_ROOT) return KVGOV_E_INVAL;
  if (n > 0 && (!tok_offsets || !blk_offsets)) return KVGOV_E_INVAL;
  if ((n_tokens > 0 && !tokens) || (n_blocks > 0 && !hashes)) return KVGOV_E_INVAL;
  if (mode == KVGOV_ROOT && n > 0 && (!principal || !salts || P <= 0)) return KVGOV_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(tokens) & 3) || (reinterpret_cast<uintptr_t>(hashes) & 3) ||
      (reinterpret_cast<uintptr_t>(salts) & 3))
    return KVGOV_E_INVAL;
  const int rc = radix_check(x);
  if (rc != KVGOV_OK) return rc;
  a = RadixArgs{};
  a.t = x->blocks->view;
  a.e = x->edges;
  a.tokens = tokens;
  a.n_tokens = n_tokens;
  a.tok_offsets = tok_offsets;
  a.n = n;
  a.principal = principal;
  a.salts = mode == KVGOV_ROOT ? salts : nullptr;
  a.P = P;
  a.zero_root = x->zero_root;
  a.hashes = hashes;
  a.blk_offsets = blk_offsets;
  a.n_blocks = n_blocks;
  return KVGOV_OK;
}

}  // namespace

extern "C" {

int kvgov_radix_create(int32_t log2_block_slots, int32_t log2_edge_slots, kvgov_radix **out) {
  if (!out || log2_block_slots < KVGOV_MIN_LOG2_SLOTS || log2_block_slots > kMaxLog2Radix ||
      log2_edge_slots < KVGOV_MIN_LOG2_SLOTS || log2_edge_slots > kMaxLog2Radix)
    return KVGOV_E_INVAL;
  *out = nullptr;
  kvgov_radix *x = new (std::nothrow) kvgov_radix();
  if (!x) return KVGOV_E_NOMEM;
  if (hipGetDevice(&x->device) != hipSuccess) {
    delete x;
    return KVGOV_E_HIP;
  }
  int rc = kvgov_cache_create(log2_block_slots, &x->blocks);
  if (rc != KVGOV_OK) {
    delete x;
    return rc;
  }
  x->edge_slots = (int64_t)1 << log2_edge_slots;
  x->edges.mask = (uint64_t)x->edge_slots - 1;
  void *keys = nullptr, *meta = nullptr, *zero = nullptr;
  if (hipMalloc(&keys, (size_t)x->edge_slots * 8) != hipSuccess ||
      hipMalloc(&meta, sizeof(RadixMeta)) != hipSuccess || hipMalloc(&zero, 32) != hipSuccess) {
    if (keys) (void)hipFree(keys);
    if (meta) (void)hipFree(meta);
    if (zero) (void)hipFree(zero);
    kvgov_cache_destroy(x->blocks);
    delete x;
    return KVGOV_E_NOMEM;
  }
  x->edges.keys = static_cast<unsigned long long *>(keys);
  x->edges.meta = static_cast<RadixMeta *>(meta);
  x->zero_root = static_cast<uint8_t *>(zero);
  rc = hipMemset(zero, 0, 32) == hipSuccess ? KVGOV_OK : KVGOV_E_HIP;
  if (rc == KVGOV_OK) rc = enqueue_edge_clear(x, nullptr);
  if (rc == KVGOV_OK && hipStreamSynchronize(nullptr) != hipSuccess) rc = KVGOV_E_HIP;
  if (rc != KVGOV_OK) {
    kvgov_radix_destroy(x);
    return rc;
  }
  *out = x;
  return KVGOV_OK;
}

int kvgov_radix_destroy(kvgov_radix *x) {
  if (!x) return KVGOV_OK;
  int rc = KVGOV_OK;
  if (hipDeviceSynchronize() != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(x->edges.keys) != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(x->edges.meta) != hipSuccess) rc = KVGOV_E_HIP;
  if (hipFree(x->zero_root) != hipSuccess) rc = KVGOV_E_HIP;
  const int rb = kvgov_cache_destroy(x->blocks);
  if (rc == KVGOV_OK) rc = rb;
  delete x;
  return rc;
}

int kvgov_radix_clear(kvgov_radix *x, void *stream) {
  if (!x) return KVGOV_E_INVAL;
  int rc = radix_check(x);
  if (rc != KVGOV_OK) return rc;
  rc = kvgov_cache_clear(x->blocks, stream);
  if (rc != KVGOV_OK) return rc;
  return enqueue_edge_clear(x, as_stream(stream));
}

int kvgov_radix_insert(kvgov_radix *x, const int32_t *tokens, int64_t n_tokens,
                       const int64_t *tok_offsets, int32_t n, const int32_t *principal,
                       const uint8_t *salts, int32_t P, int32_t mode, const uint8_t *hashes,
                       const int64_t *blk_offsets, int64_t n_blocks, void *stream) {
  RadixArgs a;
  int rc = radix_args(x, tokens, n_tokens, tok_offsets, n, principal, salts, P, mode, hashes,
                      blk_offsets, n_blocks, a);
  if (rc != KVGOV_OK || n == 0) return rc;
  hipStream_t s = as_stream(stream);
  // roots, then the full blocks' digests, then the edges below them
  kvgov_cache *c = x->blocks;
  const uint32_t epoch = c->epoch.fetch_add(1) + 1;
  if (epoch == 0xFFFFFFFFu) return KVGOV_E_UNSUPPORTED;
  const uint8_t *roots = mode == KVGOV_ROOT ? salts : x->zero_root;
  const int64_t n_roots = mode == KVGOV_ROOT ? P : 1;
  hipLaunchKernelGGL(k_radix_roots, dim3((unsigned)ceil_div(n_roots, 256)), dim3(256), 0, s,
                     c->view, roots, n_roots, epoch);
  rc = launch_status();
  if (rc != KVGOV_OK) return rc;
  rc = cache_insert_rows(c, hashes, blk_offsets, n, n_blocks, s, &a.blk_epoch);
  if (rc != KVGOV_OK) return rc;
  const int g = radix_group(n, n_blocks);
  const dim3 grid((unsigned)ceil_div((int64_t)n * g, 256)), block(256);
  switch (g) {
    case 4: hipLaunchKernelGGL(k_radix_edges<4>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(k_radix_edges<8>, grid, block, 0, s, a); break;
    case 16: hipLaunchKernelGGL(k_radix_edges<16>, grid, block, 0, s, a); break;
    case 32: hipLaunchKernelGGL(k_radix_edges<32>, grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL(k_radix_edges<64>, grid, block, 0, s, a); break;
  }
  return launch_status();
}

int kvgov_radix_match(kvgov_radix *x, const int32_t *tokens, int64_t n_tokens,
                      const int64_t *tok_offsets, int32_t n, const int32_t *principal,
                      const uint8_t *salts, int32_t P, int32_t mode, const uint8_t *hashes,
                      const int64_t *blk_offsets, int64_t n_blocks, int32_t *match_len,
                      void *stream) {
  RadixArgs a;
  int rc = radix_args(x, tokens, n_tokens, tok_offsets, n, principal, salts, P, mode, hashes,
                      blk_offsets, n_blocks, a);
  if (rc != KVGOV_OK) return rc;
  if (n == 0) return KVGOV_OK;
  if (!match_len) return KVGOV_E_INVAL;
  a.match_len = match_len;
  hipStream_t s = as_stream(stream);
  const int g = radix_group(n, n_blocks) > 16 ? 64 : 16;
  const dim3 grid((unsigned)ceil_div((int64_t)n * g, 256)), block(256);
  if (g == 16)
    hipLaunchKernelGGL(k_radix_match<16>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(k_radix_match<64>, grid, block, 0, s, a);
  return launch_status();
}

int kvgov_radix_stats(kvgov_radix *x, int64_t *block_nodes, int64_t *edges, void *stream) {
  if (!x || !block_nodes || !edges) return KVGOV_E_INVAL;
  int rc = radix_check(x);
  if (rc != KVGOV_OK) return rc;
  hipStream_t s = as_stream(stream);
  RadixMeta m{};
  if (hipMemcpyAsync(&m, x->edges.meta, sizeof m, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return KVGOV_E_HIP;
  int64_t e = 0;
  for (int i = 0; i < kCounterLanes; ++i) e += (int64_t)m.n_edges[i];
  *edges = e;
  rc = kvgov_cache_count(x->blocks, block_nodes, stream);
  if (rc != KVGOV_OK) return rc;
  return m.status;
}

}  // extern "C"
