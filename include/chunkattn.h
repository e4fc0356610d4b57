/*
 * chunkattn.h - C ABI of an MI355X (gfx950) library for decode-phase
 * self-attention over a prefix-aware, chunked KV cache, computed with the
 * two-phase partition of ChunkAttention (arXiv 2402.15220).
 *
 * Paper passages the calls follow:
 *   - Section 3.1 (PAKV): the cache is a forest whose nodes are chunks of
 *     up to c tokens with their K and V rows. Joining adds a root-to-leaf
 *     path after looking up the longest cached prefix; leaving deletes the
 *     sequence's path; a decode step adds one token to each sequence's last
 *     chunk, or a fresh child chunk once that one has no room. Chunk storage
 *     is recycled through a free list.
 *   - Section 3.2 (TPP): attention for the last token of every live sequence,
 *     Q in R^{b x d} per head (Algorithms 1 and 2, Eqn 1 and Eqn 2).
 *   - Section 3.3: the kernel context (chunk, first and last covered query
 *     row) is generated from the tree on the host and copied to the device
 *     lazily, only when the tree structure changes.
 *   - Section 3.2, prefill: a prefix lookup reports how many leading tokens
 *     are already cached so their K/V need not be recomputed.
 *
 * Conventions for every call:
 *   - Return value: CA_OK (0) or a negative ca_status, and ca_last_error()
 *     returns a message for this thread. On failure nothing observable
 *     changes (tree, tables, pool contents and slot ownership stay as they
 *     were), with two exceptions: after CA_ERR_HOST the cache's host state
 *     may be partly updated and the cache must be destroyed; after
 *     CA_ERR_DEVICE from ca_insert, ca_extend or ca_append_batch the tree
 *     change is kept but its K/V copies may not have been enqueued (HIP
 *     launch errors are normally sticky, so the cache should be destroyed
 *     too). No C++ exception leaves the library.
 *   - A cache is not thread-safe. All device work of a cache is enqueued on
 *     the hipStream_t passed to the call; callers must use one stream per
 *     cache, which also makes slot reuse after ca_remove safe (later writes
 *     are stream-ordered after earlier reads).
 *   - "host" pointers are read synchronously before the call returns;
 *     "device" pointers must stay valid until the enqueued work completes.
 *   - Tree row order: the query rows q and output rows o are ordered as the
 *     sequences appear in a depth-first walk of the tree (children by
 *     ascending first token; sequences that end at a node, by ascending id,
 *     before that node's children). ca_seq_order() returns that order. The
 *     rows covered by any chunk are then contiguous (Section 3.1).
 */
#ifndef CHUNKATTN_H
#define CHUNKATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ca_cache ca_cache; /* opaque, owned by the library */

typedef enum {
  CA_OK = 0,
  CA_ERR_INVALID = -1,   /* bad argument: null pointer, n < 1, negative token, bad shape */
  CA_ERR_NOMEM = -2,     /* the chunk pool cannot supply the slots the call needs */
  CA_ERR_NOT_FOUND = -3, /* unknown sequence id */
  CA_ERR_EXISTS = -4,    /* sequence id already live */
  CA_ERR_DEVICE = -5,    /* a HIP call failed; message holds hipGetErrorString */
  CA_ERR_WORKSPACE = -6, /* workspace null or smaller than ca_workspace_size */
  CA_ERR_HOST = -7       /* a host memory allocation inside the library failed */
} ca_status;

typedef enum { CA_FP16 = 0, CA_FP32 = 1 } ca_dtype;

/*
 * Cache configuration (Section 3.1: chunk size c; the experiments use h=32,
 * d=128, c=64, FP16).
 *   chunk_size  c >= 1 tokens per chunk
 *   num_heads   H >= 1
 *   head_dim    d in {64, 128}
 *   dtype       element type of K, V, q and o
 *   num_slots   number of chunk slots in each pool (>= 1)
 *   k_pool, v_pool  caller-owned device buffers, 16-byte aligned. The K rows
 *               of chunk slot s, head h are the c*d contiguous elements at
 *               k_pool + s*slot_stride + h*head_stride (row-major [c][d]);
 *               V likewise from v_pool. The library writes only rows it
 *               owns and never frees the pools.
 *               Both NULL: a table-only cache that keeps the tree and its
 *               tables but stores no K/V (k/v arguments must then be NULL and
 *               ca_attention is refused). Used to exercise the host tree
 *               without a GPU.
 *   slot_stride, head_stride  in elements; 0 means the dense layout
 *               [slot][head][c][d] (head_stride = c*d, slot_stride = H*c*d).
 *               head_stride >= c*d, slot_stride >= (H-1)*head_stride + c*d,
 *               both multiples of 16 bytes; K and V tiles must not overlap.
 *               Each pool spans (num_slots-1)*slot_stride + (H-1)*head_stride
 *               + c*d elements. Example: the interleaved layout
 *               [slot][head][K|V][c][d] in one buffer is v_pool = k_pool + c*d,
 *               head_stride = 2*c*d, slot_stride = 2*H*c*d.
 */
typedef struct {
  int32_t chunk_size;
  int32_t num_heads;
  int32_t head_dim;
  ca_dtype dtype;
  int64_t num_slots;
  void* k_pool;
  void* v_pool;
  int64_t slot_stride;
  int64_t head_stride;
} ca_config;

/*
 * Host views of the canonical kernel-context tables (Section 3.3, Figure 2;
 * ranges are half-open [begin, end), Figure 2 prints the end inclusively).
 * Node index = breadth-first level order, children by ascending first token.
 *   row_seq[B]          sequence id of each query row
 *   node_*[n_nodes]     slot, token count, covered rows [row_begin,row_end),
 *                       parent node (-1 for a tree root), start position of
 *                       the node's first token within its sequences
 *   shr_node[n_shared]  nodes covered by >= 2 rows (Algorithm 1's chunks)
 *   shr_part_base[n_shared]  running sum of their row counts: partial result
 *                       (node, row r) has index shr_part_base + r - row_begin
 *   priv_ptr[B+1], priv_node[]  per row, private nodes root -> leaf
 *                       (Algorithm 2's chunks C_{k+1..l})
 *   shr_ptr[B+1],  shr_part[]   per row, partial indices of its shared nodes,
 *                       root -> leaf (Algorithm 2's partials C_1..C_k)
 * Arrays are owned by the cache and valid until its next mutating call.
 */
typedef struct {
  int64_t B, n_nodes, n_shared;
  const int64_t* row_seq;
  const int32_t *node_slot, *node_len, *node_row_begin, *node_row_end, *node_parent,
      *node_start_pos;
  const int32_t *shr_node, *shr_part_base;
  const int32_t *priv_ptr, *priv_node, *shr_ptr, *shr_part;
} ca_tables;

/* Create a cache (Section 3.1). No device work; a HIP cache allocates its
 * small device tables (slot lengths, work lists) on the current device.
 * Errors: INVALID (c < 1, H < 1, d not 64/128, bad dtype, num_slots < 1, only
 * one of the pools given), DEVICE. *out receives the handle. */
ca_status ca_create(const ca_config* cfg, ca_cache** out);

/* Destroy; NULL is accepted. Never frees the caller's pools. Synchronises
 * nothing: the caller must have finished the cache's stream work. */
ca_status ca_destroy(ca_cache* cache);

/* Prefix lookup (Section 3.2, prefill): number of leading tokens of
 * tokens[0..n) already present in the tree. tokens: host int32, n >= 1,
 * every token >= 0. No mutation. */
ca_status ca_match(const ca_cache* cache, const int32_t* tokens, int64_t n, int64_t* matched);

/* A new sequence joins (Section 3.1): search the tree and insert its path.
 * A fully matched chunk is descended; a mismatch or the end of the sequence
 * inside a chunk splits that chunk (its tail moves to a fresh slot with its
 * K/V rows copied); the remaining tokens become new chunks of at most c
 * tokens. Spare room of a chunk that other sequences use is never filled.
 *   tokens  host int32 [n], n >= 1, each >= 0
 *   k, v    device [n][H][d] of dtype; rows < *matched are not read
 *           (NULL for a table-only cache)
 *   stream  hipStream_t for the K/V copies
 *   matched nullable out: tokens already present
 * Errors: INVALID, EXISTS, NOMEM (checked before any change), DEVICE. */
ca_status ca_insert(ca_cache* cache, int64_t seq_id, const int32_t* tokens, int64_t n,
                    const void* k, const void* v, void* stream, int64_t* matched);

/* Extend a live sequence by n >= 1 tokens (Section 3.1, decoding). If its
 * last chunk is used by it alone, that chunk is filled up to c first;
 * otherwise the tokens are matched below the last chunk as in ca_insert.
 * k, v: device [n][H][d]; rows < *matched are not read. Errors as ca_insert
 * plus NOT_FOUND. */
ca_status ca_extend(ca_cache* cache, int64_t seq_id, const int32_t* tokens, int64_t n,
                    const void* k, const void* v, void* stream, int64_t* matched);

/* One decode step: append tokens[i] to sequence seq_ids[i] for i < n_seqs,
 * in the listed order (Section 3.1: append into leaf chunks, grow a chunk
 * when full). seq_ids, tokens: host; k, v: device [n_seqs][H][d]. All or
 * nothing: NOMEM leaves every sequence unchanged. Ids must be distinct. */
ca_status ca_append_batch(ca_cache* cache, int64_t n_seqs, const int64_t* seq_ids,
                          const int32_t* tokens, const void* k, const void* v, void* stream);

/* A completed sequence leaves (Section 3.1): delete its path; chunks no
 * longer used by any sequence return to the pool (freed leaf first, reused
 * last-freed first). Chains are not merged. */
ca_status ca_remove(ca_cache* cache, int64_t seq_id);

/* Number of live sequences (B, the query rows of the next attention). */
ca_status ca_num_seqs(const ca_cache* cache, int64_t* B);

/* Tree row order: seq_ids[r] = id of the sequence whose query is row r.
 * seq_ids: host int64 with room for cap >= B entries. */
ca_status ca_seq_order(const ca_cache* cache, int64_t* seq_ids, int64_t cap);

/* Bytes of device workspace ca_attention needs for the current tree
 * (partial results of Algorithm 1 plus split partials; 0 is possible). */
ca_status ca_workspace_size(const ca_cache* cache, size_t* bytes);

/* Decode attention for every live sequence (Section 3.2, Algorithms 1 and 2):
 * chunk-first partial attention (Eqn 1) over chunks shared by >= 2 rows with
 * the covered query rows batched, sequence-first partial attention over each
 * row's own chunks, online-softmax merge (Eqn 2) and O/n.
 *   q      device [B][H][d] of dtype, tree row order (ca_seq_order)
 *   o      device [B][H][d] of dtype, written in the same order
 *   scale  softmax scale applied to q.k; 0 means 1/sqrt(d)
 *   ws     device workspace of ws_bytes >= ca_workspace_size() bytes,
 *          256-byte aligned; contents on entry are ignored
 * Uploads the kernel context first if the tree structure changed since the
 * last call (Section 3.3, lazy copy). B == 0 is a no-op.
 * Errors: INVALID (table-only cache, null q/o), WORKSPACE, DEVICE. */
ca_status ca_attention(ca_cache* cache, const void* q, void* o, float scale, void* ws,
                       size_t ws_bytes, void* stream);

/* ca_attention with q and o in the caller's row order: row i of q and o
 * belongs to sequence seq_ids[i] (host, n entries), which must list every
 * live sequence exactly once (n = ca_num_seqs). The kernels read q and write
 * o through a tree-row -> caller-row map, so no gather of q or scatter of o
 * is needed; the map is uploaded (library-owned pinned staging, on `stream`)
 * only when it differs from the previous call's. Other arguments and
 * errors as ca_attention, plus INVALID (n differs from the number of live
 * sequences, an id not live or listed twice). */
ca_status ca_attention_ordered(ca_cache* cache, const void* q, void* o, const int64_t* seq_ids,
                               int64_t n, float scale, void* ws, size_t ws_bytes, void* stream);

/* ca_attention for callers that cannot allocate memory: code being captured
 * into a HIP graph, tight serving loops, harnesses that forbid hipMalloc.
 * Same kernels, arguments (q, o in tree row order, scale) and result as
 * ca_attention, but the partial results and arrival counters live in a
 * device scratch array that is part of the library's code object: 16 MiB
 * per GPU the library is loaded on, held until the process ends. The call
 * itself allocates nothing (no hipMalloc, hipHostMalloc, hipFree, stream or
 * event creation): it clears the counters with a kernel on `stream`, then
 * launches the attention kernels.
 *   Preconditions: the kernel context must already be on the device, i.e.
 *   ca_prepare (or any attention call) after the last tree change that
 *   altered the chunk structure and after the last ca_set_tuning; appends
 *   that only fill existing chunks need nothing. Under schedule 3 one
 *   ca_attention call must have created the second stream.
 *   Limits: at most 65,536 (row, head) pairs (B * H) and 16,515,072 bytes
 *   of partials (ca_workspace_size); larger calls return CA_ERR_WORKSPACE
 *   and must use ca_attention with a caller workspace.
 *   Sharing: every call on one GPU uses that GPU's one scratch array, so
 *   calls that may overlap on one GPU (different streams, threads or
 *   caches) race and give wrong results; serialise them.
 * Errors: INVALID (table-only cache, null or misaligned q/o, bad scale,
 * context not current, schedule 3 without its stream), WORKSPACE, DEVICE.
 * B == 0 is a no-op. */
ca_status ca_attention_noalloc(ca_cache* cache, const void* q, void* o, float scale, void* stream);

/* Bring the kernel context up to date now (Section 3.3, further
 * optimizations: context generation hidden behind earlier GPU work). Builds
 * the tables and work lists for the current tree on the host and, if they
 * differ from the device copy, enqueues the upload on `stream`; a following
 * ca_attention on the same stream then only launches kernels. Call it after
 * a step's tree changes (joins, leaves, appends) and after enqueuing the GPU
 * work that precedes attention, so the host work overlaps that work. Without
 * it, ca_attention does the same lazily.
 *   uploaded  nullable out: 1 if an upload was enqueued, else 0
 * A table-only cache or an empty tree builds the host context only.
 * Errors: INVALID (null cache), DEVICE. */
ca_status ca_prepare(ca_cache* cache, void* stream, int32_t* uploaded);

/* Prefill attention with prefix reuse (Section 3.2, prefill paragraph): a
 * joining sequence's matched prefix keeps its K/V in the tree, its unmatched
 * suffix is written by ca_insert/ca_extend, and attention then runs over the
 * sequence's entire K/V. This computes it for the sequence's last n_q
 * tokens: query i (position L - n_q + i, L = the sequence's length) attends
 * causally to positions 0 .. L - n_q + i of its root-to-leaf chunks.
 *   q      device [n_q][H][d], 16-byte aligned; o the same shape, written
 *   n_q    0 <= n_q <= L (0 is a no-op); typically L - matched
 *   scale  softmax scale applied to q.k; 0 means 1/sqrt(d)
 * fp16 caches only. Enqueue on the stream of the insert/extend that wrote
 * the K/V rows. The path (chunk slots and start positions, 8 bytes per
 * chunk) travels inside the kernel arguments for up to 255 chunks; a longer
 * one is copied to the device through library-owned pinned staging.
 * Work is one block per (64 queries, head); when those blocks would leave
 * compute units idle (a short join over a long path), each block's key
 * range is cut into parts run by separate blocks, whose partial results
 * (O, m, n) are folded by Eqn 2 in a library-owned device workspace
 * (ceil(n_q / 64) * H * parts * (256 d + 512) bytes, grown on first need,
 * which synchronizes the stream once). CA_PREFILL_SPLIT=k in the
 * environment at ca_create forces k parts (1: never split); the results do
 * not depend on it beyond fp32 summation order.
 * Errors: INVALID (table-only or fp32 cache, null or misaligned q/o,
 * n_q > L), NOT_FOUND, DEVICE. */
ca_status ca_prefill_attention(ca_cache* cache, int64_t seq_id, const void* q, void* o,
                               int64_t n_q, float scale, void* stream);

/* Host views of the canonical tables for the current tree (see ca_tables).
 * Lengths reflect every call made so far. */
ca_status ca_export_tables(const ca_cache* cache, ca_tables* out);

/* Counters for tests and reports: number of kernel-context uploads so far,
 * slots in use, total slots, the attention schedule (see ca_set_tuning), the
 * chunk-first segment size of the current kernel context, and how many
 * context updates were done in place (decode growth: new private chunks at
 * the end of paths patch the per-row lists instead of rebuilding them,
 * Section 3.3). Any pointer may be NULL. With CA_CHECK_PATCH=1 in the
 * environment at ca_create, every in-place update is compared with a full
 * rebuild and a difference makes this call return INVALID. */
ca_status ca_stats(const ca_cache* cache, int64_t* uploads, int64_t* slots_used,
                   int64_t* slots_total, int32_t* schedule, int32_t* seg_chunks,
                   int64_t* patches);

/* Tuning and per-phase measurement (schedules change speed, not results).
 *   seg_chunks   shared chunks per chunk-first work item (1..64; 0 keeps the
 *                current value; -1, the default, sizes segments for about
 *                one chunk-first block per compute unit, at most 16 chunks
 *                unless the private K/V stream is long enough to hide longer
 *                chains, then up to 64). More chunks per item mean fewer
 *                partials.
 *   schedule     0: chunk-first launch, then a sequence-first launch whose
 *                items fold the chunk-first partials; 1: both phases in one
 *                launch (chunk-first items first), every item writes a
 *                partial, a merge launch finishes the rows; 2 (default): as
 *                1 but the last contributor to a row finishes it inside the
 *                launch; 3: the two phases as concurrent kernels,
 *                chunk-first on a stream owned by the cache that forks from
 *                and joins back into the caller's stream, rows finished as
 *                in 2; 4: partial-free reduction (Section 3.3, further
 *                optimizations): the workspace holds one accumulator per
 *                (sequence, head) instead of one partial per (segment, row,
 *                head); chunk-first segments fold into it in path order, one
 *                launch per position along the path (a run of shared chunks
 *                is one segment unless seg_chunks is set), then the
 *                sequence-first launch folds it and writes o; split_chunks
 *                is ignored. -1 keeps the current value.
 *   split_chunks private chunks per sequence-first work item; rows with more
 *                private chunks are split and merged by the merge epilogue
 *                (0 disables splitting, -1 keeps the current value).
 *   phase_mask   kernels ca_attention enqueues: bit 0 chunk-first, bit 1
 *                sequence-first, bit 2 merge (0 keeps the current value; the
 *                default 7 runs all). A subset is for timing one kernel in
 *                isolation and leaves o incomplete unless the other phases'
 *                results are already in the workspace.
 * Changing seg_chunks, split_chunks or schedule rebuilds the kernel context and
 * may change ca_workspace_size. Errors: INVALID. */
ca_status ca_set_tuning(ca_cache* cache, int32_t seg_chunks, int32_t split_chunks,
                        int32_t phase_mask, int32_t schedule);

/* Message of the last failed call on this thread ("" if none). */
const char* ca_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CHUNKATTN_H */
