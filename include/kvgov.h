/*
 * kvgov.h -- C ABI of libkvgov: the data-parallel hot path of KVGov's
 * HMAC-keyed namespace isolation for multi-tenant prefix caches, on AMD
 * Instinct MI355X (gfx950).
 *
 * The three steps of the path and the paper passages that define them:
 *
 *   salts        sigma_p = HMAC-SHA256(K, principal_id)         Sec. 4.1
 *   hash_chains  h_0 = H(T_0), h_j = H(h_{j-1} || T_j), with    Sec. 2.1
 *                the salt at the chain root (h_0 = H(sigma_p || T_0))   Sec. 4.1
 *                or at the divergence boundary k                         Sec. 4.2
 *                (h_k = H(sigma_p || h_{k-1} || T_k))
 *   cache        insert block hashes; lookup returns, per       Sec. 2.1;
 *                request, the number of leading blocks present  Table tab:taxonomy
 *                (first miss), i.e. the longest cached prefix   (block prefix cache)
 *
 * H is SHA-256 (FIPS 180-4).  T_j is the 64 bytes of block j: 16 int32
 * token ids, little-endian, back to back.  Only full blocks are hashed; a
 * trailing partial block is ignored.  Digests are stored as their standard
 * 32-byte big-endian serialisation.
 *
 * Conventions for every call:
 *   - Array arguments marked "device" are device pointers owned by the
 *     caller; the library never frees or keeps them.  "host" pointers are
 *     read or written before the call returns.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is
 *     enqueued on it in order; calls return without waiting unless stated.
 *   - Every call returns KVGOV_OK (0) or a negative KVGOV_E_* code.
 *     Argument errors that can be seen on the host return before anything is
 *     enqueued and have no side effects.  Errors found by a kernel (bad
 *     offsets, a principal or boundary out of range, a full table) are
 *     latched: in the caller's `status` word for the hashing calls, in the
 *     cache object for the cache calls, and reported by the next call that
 *     waits for the stream.
 *   - K and the salts are secrets: the library keeps no copy of K after
 *     kvgov_salts returns and logs nothing.
 *   - The calls allocate no device memory except kvgov_cache_create,
 *     kvgov_radix_create, and the per-stream scratch that kvgov_hash_chains
 *     and its resume variant, kvgov_cache_admit, the maintenance calls and
 *     the offset helpers use:
 *     one buffer per (device, stream) the library has seen, grown on demand
 *     (growth waits for that stream, then frees the old buffer) and held
 *     until the process ends.  A stream runs its work in order, so its
 *     buffer serves one call at a time and no memory passes between streams.
 */
#ifndef KVGOV_H
#define KVGOV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Salt placement.  NONE: unsalted chain (Sec. 2.1).  ROOT: salt in the first
 * block's message (Sec. 4.1).  BOUNDARY: salt in block k's message, blocks
 * below k unsalted and shared across principals (Sec. 4.2). */
#define KVGOV_NONE 0
#define KVGOV_ROOT 1
#define KVGOV_BOUNDARY 2

#define KVGOV_BLOCK_SIZE 16 /* tokens per block; the only size supported */
#define KVGOV_DIGEST_BYTES 32
#define KVGOV_MAX_KEY_BYTES 64    /* HMAC keys up to one SHA-256 block */
#define KVGOV_MAX_ID_BYTES 1024   /* principal id length limit */
#define KVGOV_MIN_LOG2_SLOTS 4
#define KVGOV_MAX_LOG2_SLOTS 31

#define KVGOV_OK 0
#define KVGOV_E_INVAL (-1)       /* bad argument seen on the host; nothing enqueued */
#define KVGOV_E_UNSUPPORTED (-2) /* valid but not supported (block size, key length) */
#define KVGOV_E_OFFSETS (-3)     /* kernel: offsets not monotone, out of bounds, or
                                    blk_offsets not the prefix sum of len // 16 */
#define KVGOV_E_BOUNDARY (-4)    /* kernel: boundary_tok outside [0, len] */
#define KVGOV_E_PRINCIPAL (-5)   /* kernel: principal index outside [0, P) */
#define KVGOV_E_FULL (-6)        /* kernel: no free slot for a new key */
#define KVGOV_E_HIP (-7)         /* a HIP runtime call failed */
#define KVGOV_E_NOMEM (-8)       /* device allocation failed */
#define KVGOV_E_CAPACITY (-9)    /* export buffer smaller than the key count */
#define KVGOV_E_DEVICE (-10)     /* cache used with another device current */
#define KVGOV_E_INTERNAL (-11)   /* kernel: an internal invariant failed (never expected) */
#define KVGOV_E_TOO_LARGE (-12)  /* batch above the allocation-free entry point's limit */

/* Largest batch (requests) of kvgov_hash_chains_noalloc. */
#define KVGOV_NOALLOC_MAX_REQUESTS 2097152

/* Opaque, library-owned prefix-cache table on one device. */
typedef struct kvgov_cache kvgov_cache;

/* Message for an error code (static string; never NULL). */
const char *kvgov_strerror(int code);

/* ABI version, (major << 16) | minor. */
int kvgov_version(void);

/*
 * a1 -- per-principal salts (Sec. 4.1): salts[p] = HMAC-SHA256(K, id_p).
 *
 * K            host, K_len bytes, 1 <= K_len <= 64 (RFC 2104 zero-pads K to
 *              64 bytes; longer keys return KVGOV_E_UNSUPPORTED).
 * principal_ids device, uint8 [P][id_len], row-major; id_len in [0, 1024].
 * salts        device out, uint8 [P][32].
 * Errors: KVGOV_E_INVAL (NULL pointer, P < 0, id_len out of range,
 * K_len == 0), KVGOV_E_UNSUPPORTED (K_len > 64), KVGOV_E_HIP.
 * P == 0 enqueues nothing.
 */
int kvgov_salts(const uint8_t *K, size_t K_len, const uint8_t *principal_ids,
                int32_t id_len, int32_t P, uint8_t *salts, void *stream);

/*
 * Output layout helper: blk_offsets[r] = sum_{i<r} floor(len_i / block_size)
 * with len_i = tok_offsets[i+1] - tok_offsets[i]; blk_offsets[0] = 0.
 *
 * tok_offsets  device, int64 [n + 1], non-decreasing.
 * blk_offsets  device out, int64 [n + 1].
 * status       device int32, zeroed by the caller; a negative length makes
 *              the kernel store KVGOV_E_OFFSETS there (first error wins).
 * Errors: KVGOV_E_INVAL, KVGOV_E_UNSUPPORTED (block_size != 16), KVGOV_E_HIP.
 */
int kvgov_block_offsets(const int64_t *tok_offsets, int32_t n, int32_t block_size,
                        int64_t *blk_offsets, int32_t *status, void *stream);

/*
 * a2/a3 -- chained block hashes for a ragged batch (Sec. 2.1, 4.1, 4.2).
 *
 * tokens       device, int32 [n_tokens]; request r owns
 *              tokens[tok_offsets[r] .. tok_offsets[r+1]).
 * tok_offsets  device, int64 [n + 1]; 0 <= tok_offsets[r] <= tok_offsets[r+1]
 *              <= n_tokens.
 * principal    device, int32 [n], index into `salts`; unused (may be NULL)
 *              for KVGOV_NONE.
 * salts        device, uint8 [P][32] (from kvgov_salts); unused for NONE.
 * mode         KVGOV_NONE, KVGOV_ROOT or KVGOV_BOUNDARY.
 * boundary_tok device, int32 [n], BOUNDARY only (may be NULL otherwise):
 *              the token offset of the divergence boundary, in [0, len_r];
 *              the salted block is k = boundary_tok / 16.  k = 0 equals root
 *              salting; k >= len_r / 16 salts no block (the unsalted chain).
 * block_size   must be 16.
 * blk_offsets  device, int64 [n + 1], as kvgov_block_offsets computes it.
 * hashes       device out, uint8 [n_blocks][32]; request r's block j goes to
 *              row blk_offsets[r] + j.  Rows of rejected requests are left
 *              untouched.
 * status       device int32, zeroed by the caller; kernels store the first
 *              error (KVGOV_E_OFFSETS / _PRINCIPAL / _BOUNDARY) there and skip
 *              the offending request.
 * Scratch: batches of more than two 64-request lane-pair workgroups per CU
 * (n > 128 * CUs) are ordered longest first using 4 * (4096 + n) bytes of
 * the stream's scratch (see the notes at the top).
 * Errors: KVGOV_E_INVAL, KVGOV_E_UNSUPPORTED, KVGOV_E_NOMEM, KVGOV_E_HIP;
 * KVGOV_E_INTERNAL latched in `status` if the ordering scratch held an
 * index outside the batch (never expected: it would mean the scratch was
 * overwritten during the call).
 */
int kvgov_hash_chains(const int32_t *tokens, int64_t n_tokens,
                      const int64_t *tok_offsets, int32_t n,
                      const int32_t *principal, const uint8_t *salts, int32_t P,
                      int32_t mode, const int32_t *boundary_tok, int32_t block_size,
                      const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                      int32_t *status, void *stream);

/*
 * kvgov_hash_chains for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and errors as kvgov_hash_chains; it
 * calls no hipMalloc, hipFree or allocating library routine.  The ordering
 * scratch of large batches is a fixed array inside the library, one per
 * device (4 * (4096 + KVGOV_NOALLOC_MAX_REQUESTS) bytes, about 8 MiB, held
 * until the process ends; its address is looked up on the first call on
 * each device).  Every call on a device shares that device's array, so
 * calls that overlap on one device (on different streams, or from several
 * host threads, without ordering between them) race and must not be
 * issued; calls in one stream are ordered and safe.  The histogram part is
 * cleared by a kernel at the start of each call.
 * Errors: as kvgov_hash_chains, and KVGOV_E_TOO_LARGE (before anything else
 * is checked) for n > KVGOV_NOALLOC_MAX_REQUESTS; KVGOV_E_HIP if the
 * scratch's address cannot be obtained.
 */
int kvgov_hash_chains_noalloc(const int32_t *tokens, int64_t n_tokens,
                              const int64_t *tok_offsets, int32_t n,
                              const int32_t *principal, const uint8_t *salts, int32_t P,
                              int32_t mode, const int32_t *boundary_tok, int32_t block_size,
                              const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                              int32_t *status, void *stream);

/*
 * Measurement of the chain kernel alone.  A chain call (kvgov_hash_chains,
 * _noalloc or _resume) enqueues, for large batches, the longest-first
 * ordering before its chain kernel; events recorded around the call measure
 * both.  After this call, the next chain call made by the same host thread
 * records start_event on its stream immediately before the chain kernel's
 * launch and end_event immediately after it, so that the elapsed time
 * between them is the kernel's.  The events are the caller's (hipEvent_t,
 * created with timing enabled, alive until used); the library keeps only
 * the two pointers and forgets them when that next chain call starts,
 * whatever it returns.  A call that returns before launching (an argument
 * error, n == 0) records neither event.  NULL, NULL clears a pending pair.
 * Errors: KVGOV_E_INVAL if exactly one pointer is NULL (nothing changes).
 * The chain call returns KVGOV_E_HIP if recording an event fails.
 */
int kvgov_time_next_chain_kernel(void *start_event, void *end_event);

/*
 * Chain extension (Sec. 2.1; Sec. 5.7 on multi-turn sessions, where turn
 * n+1 extends turn n exactly).  Because h_j depends only on h_{j-1}, T_j and,
 * for the salted block, sigma_p, a chain whose digests up to block j0 - 1 are
 * already known resumes at block j0 from h_{j0-1}: the result is exactly rows
 * j0 .. len_r/16 - 1 of what kvgov_hash_chains computes for the whole
 * request.  The prefix is neither read nor rehashed.
 *
 * Arguments as for kvgov_hash_chains (tokens hold each request's whole
 * sequence; only the tokens of blocks >= j0 are read; boundary_tok is the
 * whole sequence's), plus:
 * start_block  device, int32 [n]: j0 of request r, in [0, len_r / 16]
 *              (outside: KVGOV_E_OFFSETS in `status`, request skipped).
 *              j0 = 0 hashes the whole chain; j0 = len_r / 16 hashes nothing.
 * parents      device, uint8 [n][32], 4-byte aligned: h_{j0-1} of request r,
 *              read only when j0 > 0 (the row's content is then trusted; the
 *              salt, root or boundary, is already inside it when j0 is past
 *              the salted block).
 * blk_offsets  device, int64 [n + 1]: exclusive prefix sum of
 *              len_r / 16 - j0 (kvgov_resume_offsets); request r's block
 *              j0 + i goes to row blk_offsets[r] + i.
 * Errors: as kvgov_hash_chains; KVGOV_E_INVAL also for NULL start_block or
 * parents with n > 0, or misaligned parents.
 */
int kvgov_hash_chains_resume(const int32_t *tokens, int64_t n_tokens,
                             const int64_t *tok_offsets, int32_t n,
                             const int32_t *principal, const uint8_t *salts, int32_t P,
                             int32_t mode, const int32_t *boundary_tok, int32_t block_size,
                             const int32_t *start_block, const uint8_t *parents,
                             const int64_t *blk_offsets, uint8_t *hashes, int64_t n_blocks,
                             int32_t *status, void *stream);

/*
 * Output layout of kvgov_hash_chains_resume: blk_offsets[r] =
 * sum_{i<r} (floor(len_i / 16) - start_block[i]); blk_offsets[0] = 0.
 * A negative length or a start block outside [0, len_i / 16] stores
 * KVGOV_E_OFFSETS in `status` and counts as 0 blocks.  Otherwise as
 * kvgov_block_offsets; KVGOV_E_INVAL for NULL start_block with n > 0.
 */
int kvgov_resume_offsets(const int64_t *tok_offsets, const int32_t *start_block, int32_t n,
                         int32_t block_size, int64_t *blk_offsets, int32_t *status,
                         void *stream);

/*
 * a4/a5 -- the device-resident prefix-cache table (Sec. 2.1; Table
 * tab:taxonomy, block prefix cache).  Open addressing over 2^log2_slots
 * slots of 32-byte keys with full 256-bit compare; any 32-byte value is a
 * valid key.  No eviction: a key stays until kvgov_cache_clear.
 *
 * create: allocates 48 * 2^log2_slots bytes (32-byte keys, 8-byte tags,
 * 8-byte recency words) plus a small metadata block on the current device,
 * cleared.  log2_slots in [4, 31].  Errors: KVGOV_E_INVAL, KVGOV_E_NOMEM,
 * KVGOV_E_HIP.  The cache must be used with that device current
 * (KVGOV_E_DEVICE otherwise).
 */
int kvgov_cache_create(int32_t log2_slots, kvgov_cache **out);

/* Frees the table (waits for the device first).  NULL is accepted. */
int kvgov_cache_destroy(kvgov_cache *c);

/* Empties the table and its latched error, in stream order. */
int kvgov_cache_clear(kvgov_cache *c, void *stream);

/* Number of slots (host). */
int kvgov_cache_slots(const kvgov_cache *c, int64_t *slots);

/*
 * T <- T u {hashes[blk_offsets[0] .. blk_offsets[n])}.  Duplicate keys in the
 * batch and keys already present count once.
 *
 * hashes       device, uint8 [n_blocks][32].
 * blk_offsets  device, int64 [n + 1], non-decreasing, blk_offsets[n] <= n_blocks.
 * n_new        host out or NULL.  Non-NULL: the call waits for `stream` and
 *              stores the number of keys the batch added; it then returns
 *              any latched error.  NULL: nothing waits.
 * Kernel errors: KVGOV_E_OFFSETS (nothing inserted), KVGOV_E_FULL (the table
 * holds a consistent subset of the union; clear it before reuse).
 */
int kvgov_cache_insert(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                       int32_t n, int64_t n_blocks, int64_t *n_new, void *stream);

/*
 * hit_blocks[r] = the first j < len_r/16 whose key hashes[blk_offsets[r] + j]
 * is not in T, or blk_offsets[r+1] - blk_offsets[r] if every key is present.
 * Reads the table only; sees every insert enqueued before it.
 *
 * hit_blocks   device out, int32 [n].
 * Kernel errors: KVGOV_E_OFFSETS (latched; the affected rows are set to 0).
 */
int kvgov_cache_lookup(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                       int32_t n, int64_t n_blocks, int32_t *hit_blocks, void *stream);

/*
 * Admission: lookup-then-insert for a batch in one call, as a serving
 * engine's scheduler admits requests one after another (Sec. 2.1: a request
 * reuses the longest cached block prefix and the blocks it computes join the
 * cache).  Requests are taken in order r = 0 .. n-1; request r sees
 *   V_r = T  u  {every key of requests 0 .. r-1}
 * (T = the table before the call), and
 *   hit_blocks[r] = the first j whose key is not in V_r (or the row count),
 *   new_blocks[r] = the number of distinct keys of request r not in V_r,
 * and afterwards T <- T u {every key of the batch}.  Sum of new_blocks =
 * the keys the call added.  The result does not depend on how the work is
 * scheduled on the device.
 *
 * hashes, blk_offsets, n, n_blocks as for kvgov_cache_insert.
 * hit_blocks, new_blocks  device out, int32 [n].
 * n_new        host out or NULL, as for kvgov_cache_insert.
 * Scratch: 4 * n_blocks bytes of the stream's scratch (see the notes at
 * the top).
 * Kernel errors: KVGOV_E_OFFSETS (latched; outputs of the batch are not
 * meaningful, rows of requests found malformed are set to 0), KVGOV_E_FULL
 * (latched; keys that found no slot count as not visible and not new).
 * Errors: KVGOV_E_INVAL, KVGOV_E_NOMEM, KVGOV_E_UNSUPPORTED (2^32 - 1
 * insert or admit calls since the last clear), KVGOV_E_HIP.
 */
int kvgov_cache_admit(kvgov_cache *c, const uint8_t *hashes, const int64_t *blk_offsets,
                      int32_t n, int64_t n_blocks, int32_t *hit_blocks, int32_t *new_blocks,
                      int64_t *n_new, void *stream);

/*
 * Table maintenance (the paper gives none; a serving cache needs it).
 *
 * Recency, on a table that tracks it (kvgov_cache_set_recency; off after
 * create): every kvgov_cache_insert or kvgov_cache_admit call is one tick of
 * the table's clock (its call number since the last clear); each key of its
 * batch takes the tick as its stamp and the smallest row position (within
 * its request) it has in that batch as its depth.  Lookups do not change
 * recency.  Keys inserted while tracking is off rank below every tracked
 * key.  Tracking costs each insert and admission a read of the key's
 * recency word and, where it grows, an atomic.
 *
 * evict: keeps the largest set of whole (stamp, depth) classes, newest stamp
 * first and, within a stamp, shallowest depth first, that holds at most
 * max_keys keys, and removes the rest (KVGOV_E_UNSUPPORTED on a table that
 * does not track recency).  When every insert and admission passes whole
 * chains from block 0 (as kvgov_hash_chains lays them out), a chain's
 * earlier block never ranks below a later one, so the kept keys of every
 * chain form a prefix of it.  (Batches holding only a chain's suffix, such
 * as resumed chains, can leave suffix blocks ranked above their prefix;
 * lookups stay correct, stopping at the first absent block, and the
 * unreachable blocks go at a later eviction.)
 * erase: removes exactly the given keys (device, uint8 [n_keys][32]; keys not
 * in T are ignored), tracking or not.
 *
 * Both rebuild the table from the keys they keep (no tombstones: lookups
 * keep reading one key per probe), in stream order.  n_kept / n_erased: host
 * out or NULL; non-NULL waits for `stream`, stores the keys kept / the
 * distinct present keys erased, and returns any latched error.
 * Scratch: 40 * (slots + 1) bytes + 2 KiB of the stream's scratch (see the
 * notes at the top).  Errors: KVGOV_E_INVAL, KVGOV_E_NOMEM,
 * KVGOV_E_UNSUPPORTED (as above, or 2^32 - 1 calls since the last clear),
 * KVGOV_E_HIP, KVGOV_E_DEVICE; KVGOV_E_INTERNAL latched if the compaction
 * counted more keys than the table's slots (never expected).
 */
int kvgov_cache_set_recency(kvgov_cache *c, int32_t on);
int kvgov_cache_evict(kvgov_cache *c, int64_t max_keys, int64_t *n_kept, void *stream);
int kvgov_cache_erase(kvgov_cache *c, const uint8_t *keys, int64_t n_keys, int64_t *n_erased,
                      void *stream);

/*
 * Radix index (Table tab:taxonomy, radix-tree prefix cache; Sec. 3.5: it
 * reports the matched prefix length in tokens, finer than whole blocks;
 * Sec. 4.1: sigma_p as the root node gives each principal a disjoint tree).
 *
 * A set of token sequences per tree: one tree per principal (KVGOV_ROOT,
 * rooted at sigma_p) or one shared tree (KVGOV_NONE).  Boundary salting has
 * no radix form in the paper: KVGOV_BOUNDARY returns KVGOV_E_UNSUPPORTED.
 *   insert: adds every request's whole token sequence to its tree;
 *   match:  match_len[r] = max over sequences s in r's tree of the number of
 *           leading tokens r and s share (0 for an empty tree).
 * Internally a trie of full-block nodes (the chained digests, as in the
 * block cache) and token nodes for the first 1..15 tokens of each block
 * below its parent: match = 16 * (block depth) + (tokens matched in the next
 * block).
 *
 * create: block table of 2^log2_block_slots slots (48 B each) and edge
 * table of 2^log2_edge_slots slots (8 B each; up to 15 edges per distinct
 * block, fewer where sequences share token prefixes), both in [4, 30], on the
 * current device (which must be current for every later call:
 * KVGOV_E_DEVICE otherwise).  Errors: KVGOV_E_INVAL, KVGOV_E_NOMEM,
 * KVGOV_E_HIP.
 */
typedef struct kvgov_radix kvgov_radix;
int kvgov_radix_create(int32_t log2_block_slots, int32_t log2_edge_slots, kvgov_radix **out);

/* Frees the index (waits for the device first).  NULL is accepted. */
int kvgov_radix_destroy(kvgov_radix *x);

/* Empties both tables and the latched errors, in stream order. */
int kvgov_radix_clear(kvgov_radix *x, void *stream);

/*
 * Inserts request r = 0..n-1: tokens[tok_offsets[r] .. tok_offsets[r+1]).
 * tokens, n_tokens, tok_offsets, principal, salts, P, mode as for
 * kvgov_hash_chains (mode NONE or ROOT).
 * hashes, blk_offsets, n_blocks: the requests' chained block hashes as
 *   kvgov_hash_chains computes them for the same tokens, mode and salts
 *   (the index trusts them: other values give another index).
 * Kernel errors (latched; kvgov_radix_stats returns them): KVGOV_E_OFFSETS
 * (offsets out of range, or blk_offsets not matching len // 16; the request
 * is skipped), KVGOV_E_PRINCIPAL, KVGOV_E_FULL (a table ran out of slots;
 * clear before reuse).
 */
int kvgov_radix_insert(kvgov_radix *x, const int32_t *tokens, int64_t n_tokens,
                       const int64_t *tok_offsets, int32_t n, const int32_t *principal,
                       const uint8_t *salts, int32_t P, int32_t mode, const uint8_t *hashes,
                       const int64_t *blk_offsets, int64_t n_blocks, void *stream);

/*
 * match_len (device out, int32 [n]) as defined above; arguments as for
 * kvgov_radix_insert.  Reads the index only; sees every insert enqueued
 * before it.  Kernel errors as for insert (a skipped request gets 0).
 */
int kvgov_radix_match(kvgov_radix *x, const int32_t *tokens, int64_t n_tokens,
                      const int64_t *tok_offsets, int32_t n, const int32_t *principal,
                      const uint8_t *salts, int32_t P, int32_t mode, const uint8_t *hashes,
                      const int64_t *blk_offsets, int64_t n_blocks, int32_t *match_len,
                      void *stream);

/* Waits for `stream`; stores the number of block nodes (full-block digests
 * and roots) and of edges (token nodes), and returns the latched error. */
int kvgov_radix_stats(kvgov_radix *x, int64_t *block_nodes, int64_t *edges, void *stream);

/* Waits for `stream`; stores the number of keys in T and returns the latched
 * error, if any. */
int kvgov_cache_count(kvgov_cache *c, int64_t *n_keys, void *stream);

/*
 * Copies every key in T, in no particular order, to keys (device,
 * uint8 [cap][32]); waits for `stream`; *n_keys = number of keys in T.
 * Returns KVGOV_E_CAPACITY if that exceeds cap (the first cap keys found
 * are written).  A latched error is not returned here (kvgov_cache_count
 * returns it), so the keys of a table that reported KVGOV_E_FULL can still
 * be read.
 */
int kvgov_cache_export(kvgov_cache *c, uint8_t *keys, int64_t cap, int64_t *n_keys,
                       void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KVGOV_H */
