/*
 * hsap.h -- C ABI of libhsap: document-masked packed causal attention for one
 * sequence-parallel shard, on AMD Instinct MI355X (gfx950).
 *
 * Method (HSAP, arxiv 2606.30460):
 *   - Documents are packed into one sequence of N tokens and described by
 *     their cumulative lengths (cu_seqlens); attention stays inside each
 *     document and is causal there (sequence-packing section).
 *   - Inter-group sequence parallelism cuts the sequence into P shards of
 *     n = N / P tokens; a shard's queries meet every K/V chunk in ring order,
 *     accumulating partial results online (inter-group SP section).
 *   - SAP compiles, before any communication, which blocks of the packed
 *     causal mask carry work so that empty blocks are neither sent nor
 *     computed (compile step 1 of the SAP section); "computing" is the
 *     attention of the Q block against the K/V block at hand (instruction
 *     table of the SAP section).
 *
 * Conventions shared by every entry point:
 *   - Positions are global token indices 0..N-1.  start(t) is the first
 *     position of t's document.  Query i may attend key j iff
 *     start(i) <= j <= i.
 *   - Layout of the shards: CONTIGUOUS gives shard r positions r*n..r*n+n-1;
 *     ZIGZAG cuts N into 2P pieces of m = N/(2P) and gives shard r piece r
 *     followed by piece 2P-1-r.  A K/V chunk c has the layout of shard c.
 *   - Ring order: at ring step s shard r holds chunk (r - s) mod P.
 *   - Tensors are token-major: a row is one token, [heads, head_dim]
 *     contiguous.  "Sharded order" [P, n, H, d] stores chunk c's n rows (in
 *     that chunk's local order) at row offset c*n.
 *   - Query head h reads K/V head h / (Hq / Hkv).
 *   - bf16 is IEEE bfloat16 (1-8-7); LSE is the natural-log log-sum-exp of
 *     the scaled scores, fp32, laid out [Hq, rows].
 *   - Device pointers are caller-owned; apart from an hsap_executor (which
 *     owns its list buffers and workspace, see below) the library allocates
 *     no device memory and keeps no state between calls.  Kernels run asynchronously on
 *     the given HIP stream (NULL = default stream).  HSAP_ERR_HIP reports a
 *     launch failure only; a fault inside a kernel surfaces at the caller's
 *     next synchronisation.
 *   - Every argument is checked before anything is launched.  A failed check
 *     returns an error, launches nothing and leaves outputs untouched;
 *     hsap_last_error() then describes it.  No C++ exception crosses the ABI.
 */
#ifndef HSAP_H
#define HSAP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HSAP_OK = 0,
  HSAP_ERR_INVALID_ARG = 1,  /* malformed argument: nothing was done          */
  HSAP_ERR_CAPACITY = 2,     /* output list too small: required size returned */
  HSAP_ERR_UNSUPPORTED = 3,  /* valid, but no kernel for this shape           */
  HSAP_ERR_HIP = 4           /* the HIP runtime refused a launch              */
} hsap_status;

typedef enum { HSAP_LAYOUT_CONTIGUOUS = 0, HSAP_LAYOUT_ZIGZAG = 1 } hsap_layout;

/* A listed tile is FULL when all BM*BN of its (query, key) pairs are allowed
 * (no mask is applied) and MASKED when only some are.  Tiles with no allowed
 * pair are never listed. */
typedef enum { HSAP_TILE_FULL = 0, HSAP_TILE_MASKED = 1 } hsap_tile_kind;

/* Which tile index groups a run: HSAP_MAJOR_Q groups the tiles of one
 * (chunk, q_tile) -- the partial forward's unit of work; HSAP_MAJOR_K groups
 * the tiles of one (chunk, k_tile) -- the backward's; HSAP_MAJOR_Q_ALL groups
 * every tile of one q_tile across all chunks, in ring order -- the fused
 * forward's. */
typedef enum { HSAP_MAJOR_Q = 0, HSAP_MAJOR_K = 1, HSAP_MAJOR_Q_ALL = 2 } hsap_major;

/* One non-empty (q-tile, k-tile) block: 16-byte POD.  q_tile counts BM-row
 * tiles of the shard's local rows, k_tile counts BN-row tiles of chunk
 * `chunk`'s local rows. */
typedef struct {
  int32_t chunk;
  int32_t q_tile;
  int32_t k_tile;
  int32_t kind;   /* hsap_tile_kind */
} hsap_tile;

/* A run of tiles that share (chunk, q_tile) [HSAP_MAJOR_Q] or
 * (chunk, k_tile) [HSAP_MAJOR_K]: tiles[first .. first+count-1] of the list
 * hsap_plan_runs returns, all of one chunk.  `tile` is the shared q_tile or
 * k_tile.  `slot` is the partial-output slot the run writes: chunk +
 * P * piece, where piece > 0 only when a long q-major run was split (see
 * hsap_plan_runs); for k-major runs slot = chunk. */
typedef struct {
  int32_t slot;
  int32_t tile;
  int32_t first;
  int32_t count;
} hsap_run;

typedef struct {
  int64_t total_tokens;  /* N: tokens of one packed sequence                */
  int32_t sp_degree;     /* P >= 1                                          */
  int32_t layout;        /* hsap_layout                                     */
  int32_t shard_id;      /* r in [0, P)                                     */
  int32_t block_m;       /* BM: query rows per tile                         */
  int32_t block_n;       /* BN: key rows per tile                           */
  int32_t batch;         /* B >= 1 packed sequences per call (0 reads as 1) */
} hsap_shard_desc;

/* Batches.  B packed sequences of N tokens are concatenated: sequence b holds
 * positions b*N .. b*N+N-1, and cu_seqlens covers all B*N positions with a
 * document boundary at every b*N.  Each sequence is split P ways by the
 * layout; shard (or chunk) x holds n = N/P positions of every sequence, and
 * its local rows are b*n + l (row l of sequence b).  Every per-shard array
 * below therefore has B*n rows, doc_start has B*N entries, and no tile pairs
 * rows of two sequences.  With B = 1 this is the single packed sequence. */

typedef struct {
  hsap_shard_desc shard;
  int32_t chunk_id;      /* K/V chunk of hsap_partial_attn_fwd / _bwd; the
                            run-based entry points read the chunk of each tile
                            and ignore this field                            */
  int32_t heads_q;       /* Hq                                              */
  int32_t heads_kv;      /* Hkv, divides Hq                                 */
  int32_t head_dim;      /* d: 64 or 128                                    */
  float softmax_scale;   /* multiplies q.k; 1/sqrt(d) in the paper's formula */
} hsap_attn_desc;

/* Largest number of partials hsap_lse_merge combines in one call. */
#define HSAP_MAX_MERGE_PARTS 64

/* Human-readable name of a status code (static storage). */
const char* hsap_status_string(hsap_status status);

/* Description of the last error returned on the calling thread ("" if none). */
const char* hsap_last_error(void);

/*
 * hsap_plan -- host planner: the non-empty tiles of one shard against every
 * chunk, in canonical order.  Compile step 1 of the SAP section partitions
 * the packed causal mask into per-rank blocks by their attention pattern;
 * this does the same per (BM x BN) tile.
 *
 *   cu_seqlens   host int32 [num_docs + 1]: 0 = cu[0] <= cu[1] <= ... <=
 *                cu[num_docs] = N.  Zero-length documents are allowed.
 *   shard        N, P, layout, r, BM, BN.  Requires N % P == 0 (CONTIGUOUS)
 *                or N % 2P == 0 (ZIGZAG), BM and BN dividing n (ZIGZAG: n/2)
 *                and N < 2^31.
 *   tiles        host [capacity] or NULL.  On success holds *num_tiles tiles
 *                ordered by ring step, then q_tile, then k_tile.
 *   num_tiles    out: number of non-empty tiles (also on HSAP_ERR_CAPACITY).
 *   step_offsets host int64 [P + 1] or NULL: tiles of ring step s are
 *                tiles[step_offsets[s] .. step_offsets[s+1]-1].
 *   useful_pairs host int64 [P] or NULL: allowed (query, key) pairs per ring
 *                step (per head).
 * Returns HSAP_ERR_CAPACITY (with *num_tiles, step_offsets and useful_pairs
 * filled) when tiles is NULL or capacity < *num_tiles: call again with room.
 */
hsap_status hsap_plan(const int32_t* cu_seqlens, int32_t num_docs, const hsap_shard_desc* shard,
                      hsap_tile* tiles, int64_t capacity, int64_t* num_tiles,
                      int64_t* step_offsets, int64_t* useful_pairs);

/*
 * hsap_plan_runs -- group a canonical tile list into runs of work for the
 * kernels (host).  Not in the paper: it is this library's scheduling of the
 * planner's list onto workgroups.
 *
 *   tiles, num_tiles  the list hsap_plan returned for `shard`.
 *   major        HSAP_MAJOR_Q: runs of one (chunk, q_tile).  A q-tile with
 *                more than max_run_tiles tiles in a chunk is cut into
 *                ceil(count / max_run_tiles) pieces of near-equal length,
 *                piece i writing slot chunk + P * i (split-K: the LSE merge
 *                combines the pieces like chunks).  Every slot a chunk uses
 *                has a run for every q_tile -- count 0 where the q_tile has
 *                no tile there -- so the forward writes LSE = -inf for every
 *                row of a used slot it does not compute.  Chunks without
 *                tiles get no runs.  sorted_tiles is the input order.
 *                HSAP_MAJOR_K: one run per (chunk, k_tile) that has tiles,
 *                slot = chunk; sorted_tiles is ordered by ring step, k_tile,
 *                q_tile.  max_run_tiles is ignored.
 *                HSAP_MAJOR_Q_ALL: one run per q_tile over all chunks (every
 *                q_tile has one: a query always attends itself), slot = 0;
 *                sorted_tiles is ordered by q_tile, ring step, k_tile.
 *                max_run_tiles is ignored.
 *   max_run_tiles  longest q-major run; <= 0 means no splitting.
 *   sorted_tiles host [num_tiles] out: the tiles the runs index.
 *   runs         host [capacity] or NULL, out: ordered by count descending
 *                (longest work first), ties by ring step, tile, slot.
 *   num_runs     out: number of runs (also on HSAP_ERR_CAPACITY).
 *   num_slots    out, nullable: 1 + the largest slot used, i.e. the number
 *                of [n, Hq, d] partial slots the forward's outputs need.
 */
hsap_status hsap_plan_runs(const hsap_shard_desc* shard, const hsap_tile* tiles, int64_t num_tiles,
                           int32_t major, int32_t max_run_tiles, hsap_tile* sorted_tiles, hsap_run* runs,
                           int64_t capacity, int64_t* num_runs, int32_t* num_slots);

/*
 * hsap_split_length -- a max_run_tiles for hsap_plan_runs (host).  Returns 0
 * (no split) unless the longest possible q-major run exceeds the average
 * work per resident workgroup, num_tiles * heads_q / resident_workgroups;
 * then that average, rounded up, floored at 4 tiles and at a quarter of a
 * chunk's k-tiles (at most four pieces).  Returns -1 for invalid arguments.
 */
int32_t hsap_split_length(const hsap_shard_desc* shard, int64_t num_tiles, int32_t heads_q,
                          int32_t resident_workgroups);

/*
 * hsap_fwd_resident_workgroups -- workgroups of the bf16 partial forward that
 * fit on the current device at once for the shapes in `desc`: the HIP
 * runtime's occupancy of the kernel hsap_partial_attn_fwd_runs dispatches for
 * (head_dim, BM, BN) (its registers, LDS and workgroup size), times the
 * device's compute units -- the resident_workgroups of hsap_split_length.
 * Not in the paper (scheduling of this library's kernels).
 *   out  host int32, written (0 on failure).
 * Returns HSAP_ERR_UNSUPPORTED for shapes without a forward kernel and
 * HSAP_ERR_HIP when the device cannot be queried.
 */
hsap_status hsap_fwd_resident_workgroups(const hsap_attn_desc* desc, int32_t* out);

/*
 * hsap_load_matrix -- the size of every rank block of the packed sequence
 * (host): for each shard r (query rows) and chunk c (key rows), the number of
 * non-empty tiles and of allowed (query, key) pairs per head that hsap_plan
 * finds for shard r in chunk c.  These are the blocks of compile step 1 of
 * the SAP section, over all ranks; their sizes are what compile step 2
 * balances.
 *   cu_seqlens  host int32 [num_docs + 1] (rules of hsap_plan).
 *   shard       N, P, layout, BM, BN; shard_id is ignored (every shard).
 *   tiles       host int64 [P * P] or NULL: tiles[r * P + c].
 *   pairs       host int64 [P * P] or NULL: pairs[r * P + c]; each row sums
 *               to sum over shard r's queries i of (i - start(i) + 1).
 *   At least one of tiles and pairs must be given.
 */
hsap_status hsap_load_matrix(const int32_t* cu_seqlens, int32_t num_docs, const hsap_shard_desc* shard,
                             int64_t* tiles, int64_t* pairs);

/*
 * hsap_balance -- the Q-transfer rebalance of rank blocks over ranks (host).
 * The workload balancing of compile step 2 (SAP section) follows LightSeq's
 * scheduling, and HSAP balances InterSP groups by additionally transferring
 * Q blocks; this is one concrete rule for it.  Block (r, c), r != c, runs
 * either on rank r once chunk c's K/V reach it (the ring) or on rank c, the
 * chunk's owner, once Q_r reaches it (its partial O and LSE then go back to
 * r for the merge).  Diagonal and empty blocks stay on r.  Starting from the
 * ring (every block on r), the most loaded rank (lowest index among equals)
 * hands one of its blocks to the block's other eligible rank while the
 * receiver stays below the giver's load, choosing the move that leaves the
 * smaller maximum of the two loads (equal: lower r, then lower c); it stops
 * when the most loaded rank has no such move.  The result is never worse
 * than the ring.
 *   cost       host int64 [P * P], >= 0: cost[r * P + c] of block (r, c),
 *              e.g. its tiles from hsap_load_matrix.
 *   exec_rank  host int32 [P * P] out: r or c, the rank computing the block.
 *   load       host int64 [P] out or NULL: the summed cost per rank.
 */
hsap_status hsap_balance(int32_t sp_degree, const int64_t* cost, int32_t* exec_rank, int64_t* load);

/* Instruction set of the per-rank programs (instruction table of the SAP
 * section): send / receive of a tensor to / from a peer, computing one rank
 * block, and the local combination of results -- the copy-and-rescale of
 * partial outputs (one merge of all of a shard's parts) in the forward, the
 * accumulation of gradient parts (one sum per gradient) in the backward.
 * Tensors: q (a shard's Q), kv (a chunk's K and V), o (a block's partial O
 * and LSE), dq (a block's dQ part), dkv (a block's dK and dV parts), do (a
 * shard's dO with its final LSE and delta = rowsum(dO o O)). */
typedef enum { HSAP_OP_SEND = 0, HSAP_OP_RECV = 1, HSAP_OP_COMPUTE = 2, HSAP_OP_MERGE = 3 } hsap_op_kind;
typedef enum {
  HSAP_T_NONE = -1,
  HSAP_T_Q = 0,
  HSAP_T_KV = 1,
  HSAP_T_O = 2,
  HSAP_T_DQ = 3,
  HSAP_T_DKV = 4,
  HSAP_T_DO = 5
} hsap_tensor_kind;

/* One instruction, 32-byte POD.  Buffers of a rank: its own Q shard and K/V
 * chunk; two receive slots each for Q and K/V; two result slots for the
 * partials it computes for other shards; one part slot per chunk with tiles
 * of its own shard (part index = that chunk's rank among them).
 *   SEND     tensor (Q: shard; KV: chunk; O: shard and chunk) to `peer`;
 *            in_slot = result slot for O, -1 for the own Q / K/V.
 *   RECV     the matching tensor from `peer` into out_slot (receive slot for
 *            Q and K/V, part index for O).
 *   COMPUTE  block (shard, chunk): Q is the own shard or receive slot
 *            in_slot, K/V the own chunk or receive slot in_slot (-1 when
 *            both are local); the partial goes to part out_slot (own shard)
 *            or result slot out_slot (another shard's).
 *   MERGE    the out_slot parts of the own shard into its output. */
typedef struct {
  int32_t op;        /* hsap_op_kind */
  int32_t tensor;    /* hsap_tensor_kind (SEND, RECV) */
  int32_t peer;      /* SEND: destination rank; RECV: source rank; else -1 */
  int32_t stage;
  int32_t shard;     /* query shard of the block, Q or O; -1 for K/V */
  int32_t chunk;     /* chunk of the block, K/V or O; -1 for Q */
  int32_t in_slot;
  int32_t out_slot;
} hsap_op;

/*
 * hsap_emit_forward -- the per-rank instruction lists of the forward pass
 * (host), the jitted code generation of the SAP section: each rank computes
 * the non-empty blocks assigned to it one per stage -- its diagonal block
 * first, then by ring step (r - c) mod P, shard, chunk (a rank without a
 * diagonal block starts at stage 1).  Inputs arrive one stage ahead straight
 * from their owner into receive slot (stage % 2); a block computed for another
 * shard returns its partial one stage later; the last stage returns the last
 * partials and merges.  Within a stage a rank lists its sends and receives
 * (ordered by peer, send before receive, tensor, shard, chunk), then its
 * computation, then the merge.  Every SEND has the matching RECV at the same
 * stage of the peer's list, so each stage's transfers form one batched
 * point-to-point group.
 *   block_tiles   host int64 [P * P]: non-empty tiles of block (r, c)
 *                 (hsap_load_matrix); empty blocks are not computed.
 *   exec_rank     host int32 [P * P]: r or c for every non-empty block
 *                 (hsap_balance, or r everywhere for the plain ring).
 *   ops           host [capacity] or NULL: rank e's instructions are
 *                 ops[rank_offsets[e] .. rank_offsets[e+1]-1], by stage.
 *   rank_offsets  host int64 [P + 1] out (also on HSAP_ERR_CAPACITY).
 *   num_stages    out: stages of the program (compute stages + 1).
 */
hsap_status hsap_emit_forward(int32_t sp_degree, const int64_t* block_tiles, const int32_t* exec_rank, hsap_op* ops,
                              int64_t capacity, int64_t* rank_offsets, int32_t* num_stages);

/*
 * hsap_emit_backward -- the per-rank instruction lists of the backward pass
 * (host), the jitted code generation of the SAP section for the gradient
 * messages of its instruction table (dq, dkv, do): every non-empty block is
 * computed on the rank that computed its forward (exec_rank), at the same
 * stage as in hsap_emit_forward.
 *   Ring block (r, c), c != r, on rank r: K/V of chunk c arrive from rank c
 *     one stage ahead (receive slot stage % 2); the block's dQ part stays on
 *     r; its dK/dV part goes to result slot stage % 2 and is sent to rank c
 *     one stage later (SEND/RECV of tensor DKV, shard r, chunk c).
 *   Transferred block (r, c), r != c, on rank c: Q and dO (with the final
 *     LSE and delta of shard r) arrive from rank r one stage ahead (two
 *     receives into slot stage % 2); the dK/dV part stays on c; the dQ part
 *     goes to result slot stage % 2 and is sent to rank r one stage later
 *     (tensor DQ).
 *   Diagonal block (e, e): local data only; both parts stay on e.
 * COMPUTE: in_slot = the receive slot of the block's inputs and out_slot =
 * the result slot of the part that leaves the rank (both -1 for a diagonal
 * block).  Parts that stay, and every received part, are indexed as
 * RECV.out_slot is: dQ part part(r, c) = rank of chunk c among the chunks
 * with a non-empty block of shard r; dK/dV part kpart(c, r) = rank of shard r
 * among the shards with a non-empty block in chunk c.  In the last stage a
 * rank with dQ parts lists MERGE (tensor DQ, shard e, out_slot = the number
 * of parts): the sum of its dQ parts in part order; and one with dK/dV parts
 * MERGE (tensor DKV, chunk e, out_slot = the number of parts) likewise.  The
 * order inside a stage and the matching of sends and receives are those of
 * hsap_emit_forward; arguments, output layout and errors as there.
 */
hsap_status hsap_emit_backward(int32_t sp_degree, const int64_t* block_tiles, const int32_t* exec_rank, hsap_op* ops,
                               int64_t capacity, int64_t* rank_offsets, int32_t* num_stages);

/*
 * hsap_doc_start -- device int32 [total_tokens]: start(t) for every position
 * t (total_tokens = B*N for a batch).
 *   cu_seqlens  device int32 [num_docs + 1] (same rules as hsap_plan; the
 *               device copy is not re-validated).
 */
hsap_status hsap_doc_start(const int32_t* cu_seqlens, int32_t num_docs, int64_t total_tokens,
                           int32_t* doc_start, void* hip_stream);

/*
 * hsap_shard_gather -- place a global-order tensor into sharded order (the
 * in-memory stand-in for scattering a sequence over P ranks).
 *   src  device [B*N rows] in global token order; dst device [P, B*n rows].
 *   row_bytes  bytes per token row, a multiple of 16; src and dst 16-byte
 *              aligned.  Uses shard->total_tokens, sp_degree, layout and
 *              batch only.
 */
hsap_status hsap_shard_gather(const hsap_shard_desc* shard, const void* src, void* dst,
                              int64_t row_bytes, void* hip_stream);

/*
 * hsap_partial_attn_fwd -- "computing" of the SAP instruction table for the
 * forward: shard r's queries against K/V chunk c = desc->chunk_id, one
 * partial output and log-sum-exp (the attention equation of the inter-group
 * SP section restricted to the packing mask and to chunk c's keys), for the
 * non-empty tiles that hsap_plan listed for that chunk.
 *
 *   desc       shard (N, P, layout, r, BM, BN), chunk_id c in [0, P), heads,
 *              head_dim, softmax scale.  Shapes as hsap_partial_attn_fwd_runs.
 *   q          device bf16 [n, Hq, d]: shard r's queries, local row order.
 *   k, v       device bf16 [P, n, Hkv, d] sharded order; only chunk c's rows
 *              are read (a caller holding chunk c alone may pass the address
 *              chunk 0 would have, k_c - c * n * Hkv * d).
 *   doc_start  device int32 [N] from hsap_doc_start.
 *   tiles      device hsap_tile [num_tiles]: chunk c's tiles in hsap_plan's
 *              order (the ring step's range tiles[step_offsets[s] ..
 *              step_offsets[s+1]-1] with c = (r - s) mod P): q_tile ascending,
 *              then k_tile, every tile's chunk equal to c.  The kernels trust
 *              the list (they index with its q_tile / k_tile values) and find
 *              each q-tile's tiles in it by search; NULL when num_tiles = 0.
 *   num_tiles  0 .. 2^31 - 1.
 *   o_part     device fp32 [n, Hq, d], 16-byte aligned: rows with an allowed
 *              key in chunk c receive the normalised partial output; rows
 *              without one are undefined and must not be read.
 *   lse_part   device fp32 [Hq, n]: every row written; -inf where the row has
 *              no allowed key in chunk c (always for q-tiles without a tile).
 * One launch of (n / BM) x Hq workgroups on `stream`; HSAP_ERR_INVALID_ARG
 * for a bad chunk_id, count or pointer, HSAP_ERR_UNSUPPORTED for shapes
 * without a kernel, both before anything is launched.  Same bits as
 * hsap_partial_attn_fwd_runs over the unsplit q-major runs of chunk c.
 */
hsap_status hsap_partial_attn_fwd(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                  const int32_t* doc_start, const hsap_tile* tiles, int64_t num_tiles,
                                  float* o_part, float* lse_part, void* hip_stream);

/*
 * hsap_partial_attn_bwd -- "computing" for the backward, on the same tile
 * list: the gradients of hsap_partial_attn_fwd's partial with P = exp(s - LSE)
 * recomputed from the shard's final LSE (the backward of the attention
 * equation; its dq and dkv results are the dq / dkv messages of the SAP
 * instruction table):
 *   dV_c += P^T dO,  dS = P o (dO V_c^T - delta),
 *   dQ   += scale dS K_c,  dK_c += scale dS^T Q,
 * dK/dV summed over the query heads of each K/V head.
 *
 *   desc, q, k, v, doc_start, tiles, num_tiles  as for hsap_partial_attn_fwd
 *              (chunk c = desc->chunk_id).  Shapes as
 *              hsap_partial_attn_bwd_runs; additionally n / BM <= 2048
 *              (the dK/dV kernel gathers each k-tile's q-tiles in LDS).
 *   d_o        device bf16 [n, Hq, d] (shard r, local rows).
 *   lse        device fp32 [Hq, n]: the shard's final (merged) forward LSE.
 *   delta      device fp32 [Hq, n] from hsap_attn_bwd_preprocess.
 *   dq_acc     device fp32 [n, Hq, d] (+=): every q-tile with a tile.
 *   dk_acc, dv_acc  device fp32 [P, n, Hkv, d] sharded order (+=): the rows
 *              of chunk c's k-tiles that have a tile (a caller holding chunk c
 *              alone may pass the address chunk 0 would have).
 * Two launches on `stream` (dQ: (n / BM) x Hq workgroups; dK/dV: (n / BN) x
 * Hkv workgroups, each scanning the list for its k-tile).  The caller zeroes
 * the accumulators once; one call per chunk of a ring accumulates dQ over the
 * ring.  Errors as for hsap_partial_attn_fwd.  For the gradients of every
 * chunk at once, the run-based entry points below avoid the per-k-tile scans.
 */
hsap_status hsap_partial_attn_bwd(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                  const void* d_o, const float* lse, const float* delta, const int32_t* doc_start,
                                  const hsap_tile* tiles, int64_t num_tiles, float* dq_acc, float* dk_acc,
                                  float* dv_acc, void* hip_stream);

/*
 * hsap_partial_attn_fwd_runs -- "computing" for the forward: for every run (slot,
 * q_tile t), the queries of q-tile t of shard r against the run's k-tiles of
 * one chunk, producing that slot's partial output and log-sum-exp (attention
 * equation of the inter-group SP section restricted to the packing mask).
 *
 *   desc       shard layout (N, P, layout, r, BM, BN) and heads / head_dim /
 *              softmax scale.  Supported: d in {64, 128}; BM in {64, 128},
 *              or 256 with d = 128; BN in {64, 128}; Hq % Hkv == 0.
 *   q          device bf16 [n, Hq, d]: shard r's queries, local row order.
 *   k, v       device bf16 [P, n, Hkv, d]: every chunk, sharded order.  Only
 *              the rows of the chunks that the passed runs' tiles name are
 *              read, so a caller holding one received chunk c alone may pass
 *              the address that chunk 0 would have (k_c - c * n * Hkv * d).
 *   doc_start  device int32 [N] from hsap_doc_start.
 *   tiles      device hsap_tile [..]: sorted_tiles of hsap_plan_runs(MAJOR_Q).
 *   runs       device hsap_run [num_runs] from hsap_plan_runs(MAJOR_Q); any
 *              subset of them may be passed (e.g. one ring step's).
 *   o_part     device fp32 [num_slots, n, Hq, d]: for each run with count > 0,
 *              rows of q-tile t in the run's slot receive the normalised
 *              partial output over the run's allowed keys (0 for a row with
 *              none).
 *   lse_part   device fp32 [num_slots, Hq, n]: rows of q-tile t in the run's
 *              slot receive the partial LSE, -inf where the row has no
 *              allowed key among the run's tiles (always for count 0).
 *   num_slots  slots o_part and lse_part hold (>= 1); a run whose slot is not
 *              below it is skipped by the kernel.
 *   Rows of o_part whose LSE is -inf are not written when count == 0 and
 *   must not be read (hsap_lse_merge does not).  Rows outside every passed
 *   run are untouched.  tiles and runs must be the lists hsap_plan_runs made
 *   for this shard: the kernel trusts their tile indices.
 */
hsap_status hsap_partial_attn_fwd_runs(const hsap_attn_desc* desc, const void* q, const void* k,
                                  const void* v, const int32_t* doc_start, const hsap_tile* tiles,
                                  const hsap_run* runs, int64_t num_runs, float* o_part,
                                  float* lse_part, int32_t num_slots, void* hip_stream);

/*
 * hsap_attn_fwd_fused -- the partial forward and the merge in one pass: for
 * every q_tile, the queries against the listed k-tiles of every chunk in
 * ring order, with one online softmax carried across the chunks (the ring's
 * online accumulation), writing the final output directly.  This is the
 * fusion of the copy and rescale operations into the attention computation
 * that the paper's Limitations section proposes as future work.
 *
 *   desc, q, k, v, doc_start  as for hsap_partial_attn_fwd_runs (same supported
 *              shapes).
 *   tiles, runs, num_runs  device lists from hsap_plan_runs(MAJOR_Q_ALL).
 *   o_out      device bf16 [n, Hq, d] (round to nearest even).
 *   lse_out    device fp32 [Hq, n].
 *   Rows of q-tiles outside the passed runs are untouched.
 */
hsap_status hsap_attn_fwd_fused(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs,
                                int64_t num_runs, void* o_out, float* lse_out, void* hip_stream);

/*
 * hsap_quantize_fp8 -- e4m3 codes of bf16 Q or K for the fp8 score variant
 * (an extension beyond the paper's bf16 attention).  For every group g and
 * head h of x [G, rows, H, d]: amax = max |x| over rows and d; scale[g, h] =
 * amax / 448 and inv = 448 / amax (fp32 divisions; both 0 when amax = 0);
 * code = e4m3(clamp(x * inv, -448, 448)), the fp32 product rounded to nearest
 * even into the OCP e4m3 format (bias 7, largest finite value 448).  A
 * shard's Q is G = 1; the chunks' K is G = P (one scale per chunk and head).
 *   x          device bf16 [G, rows, H, d], 16-byte aligned; d a multiple
 *              of 8.
 *   codes      device uint8 [G, rows, H, d], 8-byte aligned.
 *   scale      device fp32 [G, H].
 *   workspace  device fp32 [G * H * HSAP_QUANT_SPLIT]: per-range maxima (each
 *              slice's rows are reduced in HSAP_QUANT_SPLIT ranges); caller
 *              owned, contents on entry ignored.
 * Two launches on `stream`.  NaN or infinite inputs are not handled.
 */
#define HSAP_QUANT_SPLIT 32
hsap_status hsap_quantize_fp8(const void* x, int32_t groups, int64_t rows, int32_t heads, int32_t head_dim,
                              uint8_t* codes, float* scale, float* workspace, void* hip_stream);

/*
 * hsap_quantize_fp8_noalloc -- hsap_quantize_fp8 with no workspace argument,
 * for callers that cannot allocate device memory around the call (code under
 * HIP graph capture, serving loops that forbid allocation): the per-range
 * maxima go to a scratch array of fixed size inside the library (512 KiB of
 * device memory per GPU the library runs on, held until the process ends).
 * Allocates nothing.  Same arguments, results and launches as
 * hsap_quantize_fp8 otherwise.
 *   groups * heads  at most HSAP_QUANT_NOALLOC_MAX_SLICES, else
 *                   HSAP_ERR_UNSUPPORTED before anything is launched.
 * Every call on one GPU shares that GPU's scratch array: calls that overlap
 * on one GPU (e.g. on two streams without ordering between them) race and may
 * produce wrong scales and codes; calls ordered on one stream are safe.  The
 * first call on a device looks up that device's copy of the array (with that
 * device current) and returns HSAP_ERR_HIP if the runtime cannot.
 */
#define HSAP_QUANT_NOALLOC_MAX_SLICES 4096
hsap_status hsap_quantize_fp8_noalloc(const void* x, int32_t groups, int64_t rows, int32_t heads, int32_t head_dim,
                                      uint8_t* codes, float* scale, void* hip_stream);

/*
 * hsap_partial_attn_fwd_fp8 -- hsap_partial_attn_fwd_runs with the scores taken
 * from e4m3 operands: S = (Q8 K8^T) * q_scale[h] * k_scale[c, g] /
 * sqrt-scale as in desc, i.e. the attention of the dequantised Q and K
 * (codes times scales); softmax, P V (bf16 V) and the outputs as in the bf16
 * partial forward.  Uses the 32x32x64 fp8 MFMA (twice the bf16 rate).
 *   q8        device uint8 [n, Hq, d], q_scale device fp32 [Hq]
 *             (hsap_quantize_fp8 with G = 1), 16-byte aligned.
 *   k8        device uint8 [P, n, Hkv, d], k_scale device fp32 [P, Hkv]
 *             (G = P), 16-byte aligned.
 *   v, doc_start, tiles, runs, o_part, lse_part, num_slots  as for
 *             hsap_partial_attn_fwd_runs.
 * Supported: head_dim 128; BM 64, 128 or 256; BN 64 or 128.
 */
hsap_status hsap_partial_attn_fwd_fp8(const hsap_attn_desc* desc, const uint8_t* q8, const uint8_t* k8,
                                      const void* v, const float* q_scale, const float* k_scale,
                                      const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs,
                                      int64_t num_runs, float* o_part, float* lse_part, int32_t num_slots,
                                      void* hip_stream);

/*
 * hsap_lse_merge -- online-softmax combination of partial results (the ring's
 * online accumulation, after Milakov & Gimelshein, inter-group SP section):
 *   L = m + ln sum_p exp(LSE_p - m),  m = max_p LSE_p;
 *   O = sum_p exp(LSE_p - L) O_p, skipping parts whose LSE is -inf (their O
 *   rows are never read); all -inf gives O = 0, L = -inf.
 *
 *   num_parts  1 .. HSAP_MAX_MERGE_PARTS.
 *   o_parts    HOST array of num_parts device pointers, each fp32 [n, Hq, d].
 *   lse_parts  HOST array of num_parts device pointers, each fp32 [Hq, n].
 *   o_out      device bf16 [n, Hq, d] (round to nearest even).
 *   lse_out    device fp32 [Hq, n].
 *   Supported head_dim: 64, 128.  Output pointers 16-byte aligned.
 */
hsap_status hsap_lse_merge(int32_t num_parts, const float* const* o_parts, const float* const* lse_parts,
                           int64_t n, int32_t heads_q, int32_t head_dim, void* o_out, float* lse_out,
                           void* hip_stream);

/*
 * hsap_attn_bwd_preprocess -- delta[h, i] = sum_d dO[i, h, d] * O[i, h, d]
 * (fp32 accumulation), the per-row term of the softmax backward.  The
 * backward half of each rank's per-step code receives the output gradient of
 * its query shard (the `do` message of the instruction table of the SAP
 * section) next to its own O; this is the first thing computed from them,
 * before the dq / dkv messages go back (differentiating the attention
 * equation of the inter-group SP section gives dS = P o (dP - delta)).
 *   o, d_o  device bf16 [n, Hq, d]: shard r's final output and its gradient,
 *           local row order, 16-byte aligned.
 *   delta   device fp32 [Hq, n], written (every row).
 *   n >= 0, heads_q >= 1, head_dim in {64, 128} (else HSAP_ERR_UNSUPPORTED);
 *   one launch on `stream`, nothing launched for n = 0.
 */
hsap_status hsap_attn_bwd_preprocess(const void* o, const void* d_o, int64_t n, int32_t heads_q,
                                     int32_t head_dim, float* delta, void* hip_stream);

/*
 * hsap_partial_attn_bwd_runs -- "computing" for the backward: the gradients of the
 * forward above with P = exp(s - LSE) recomputed from the final LSE:
 *   dV_c += P^T dO,  dS = P o (dO V_c^T - delta),
 *   dQ   += scale dS K_c,  dK_c += scale dS^T Q,
 * with dK/dV summed over the query heads of each K/V head.  Two kernels run
 * on the stream: one over the k-major runs (dK, dV) and one over the q-major
 * runs (dQ); either list may be empty (count 0) to skip its kernel.
 *
 *   desc, q, k, v, doc_start  as for the forward.  Supported: d = 128 with
 *              BM in {64, 128, 256} and BN in {64, 128}; d = 64 with BM in
 *              {64, 128} and BN = 64.  The q-major runs (dQ kernel) further
 *              need sp_degree <= 256 and fewer than 2^23 k-tiles per chunk
 *              (packed tile descriptors); HSAP_ERR_UNSUPPORTED otherwise,
 *              before anything is launched.
 *   d_o        device bf16 [n, Hq, d] (shard r, local rows).
 *   lse        device fp32 [Hq, n]: the merged forward LSE.
 *   delta      device fp32 [Hq, n] from hsap_attn_bwd_preprocess.
 *   tiles_k, runs_k, num_runs_k  device lists from hsap_plan_runs(MAJOR_K).
 *              k, v, dk_acc and dv_acc are read and written only in the
 *              rows of the chunks that the passed runs' tiles name, so a
 *              caller holding one chunk c alone may pass the addresses that
 *              chunk 0 would have (as for hsap_partial_attn_fwd_runs).
 *   tiles_q, runs_q, num_runs_q  device q-tile runs in which no q_tile
 *              appears twice: hsap_plan_runs(MAJOR_Q_ALL) (every chunk in
 *              one pass), or the runs of one chunk from
 *              hsap_plan_runs(MAJOR_Q) with max_run_tiles = 0 (one ring
 *              step).  A run may span several chunks.
 *   dq_acc     device fp32 [n, Hq, d] (+=).  Each run owns its q-tile's rows
 *              for the call: plain read-modify-write, no atomics (so runs
 *              sharing a q-tile, e.g. split pieces, must go to separate
 *              calls).
 *   dk_acc, dv_acc  device fp32 [P, n, Hkv, d] sharded order (+=).  Each
 *              (chunk, k_tile, K/V head) row block is owned by one
 *              workgroup: plain read-modify-write.
 *   The caller zeroes the accumulators once; concurrent calls on the same
 *   accumulators race.
 */
hsap_status hsap_partial_attn_bwd_runs(const hsap_attn_desc* desc, const void* q, const void* k,
                                  const void* v, const void* d_o, const float* lse,
                                  const float* delta, const int32_t* doc_start,
                                  const hsap_tile* tiles_k, const hsap_run* runs_k, int64_t num_runs_k,
                                  const hsap_tile* tiles_q, const hsap_run* runs_q, int64_t num_runs_q,
                                  float* dq_acc, float* dk_acc, float* dv_acc, void* hip_stream);

/*
 * hsap_attn_bwd_bf16 -- hsap_partial_attn_bwd_runs over every chunk in one pass
 * with the finalisation fused: each q-tile and each (chunk, k_tile, K/V
 * head) block has exactly one owning run, so its gradient is complete in
 * registers and stored once, as bf16 (round to nearest even), instead of
 * being added to fp32 accumulators and converted afterwards.
 *
 *   desc, q, k, v, d_o, lse, delta, doc_start  as for hsap_partial_attn_bwd_runs
 *              (same supported shapes).
 *   tiles_k, runs_k, num_runs_k  hsap_plan_runs(MAJOR_K) lists.
 *   tiles_q, runs_q, num_runs_q  hsap_plan_runs(MAJOR_Q_ALL) lists.
 *   dq         device bf16 [n, Hq, d], 8-byte aligned: the rows of every
 *              q-tile of runs_q are written (0 where a q-tile has no key).
 *   dk, dv     device bf16 [P, n, Hkv, d] sharded order: the rows of every
 *              (chunk, k_tile) with a k-major run are written; all other
 *              rows are left untouched (the caller zeroes them).
 */
hsap_status hsap_attn_bwd_bf16(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                               const void* d_o, const float* lse, const float* delta, const int32_t* doc_start,
                               const hsap_tile* tiles_k, const hsap_run* runs_k, int64_t num_runs_k,
                               const hsap_tile* tiles_q, const hsap_run* runs_q, int64_t num_runs_q, void* dq,
                               void* dk, void* dv, void* hip_stream);

/*
 * hsap_sum_parts -- out[i] = parts[0][i] + parts[1][i] + ... (fp32, added in
 * part order), stored as fp32 or as bf16 (round to nearest even).  The
 * accumulation of gradient parts in the backward's per-rank programs: a rank
 * sums the dQ parts of its shard and the dK/dV parts of its chunk that it
 * computed or received (the dq / dkv messages of the instruction table of
 * the SAP section; see hsap_emit_backward).
 *   num_parts  1 .. HSAP_MAX_MERGE_PARTS.
 *   parts      HOST array of num_parts device pointers, each fp32 [count],
 *              16-byte aligned.
 *   out        device fp32 [count] (16-byte aligned) or, with out_bf16 != 0,
 *              bf16 [count] (8-byte aligned); may not overlap a part.
 * One launch on `stream`; nothing launched for count = 0.
 */
hsap_status hsap_sum_parts(int32_t num_parts, const float* const* parts, int64_t count, void* out, int32_t out_bf16,
                           void* hip_stream);

/*
 * hsap_convert_f32_bf16 -- dst[i] = bf16(src[i]), round to nearest even
 * (finalising fp32 gradient accumulators).  count >= 0; pointers 16-byte
 * aligned when count is a multiple of 8.
 */
hsap_status hsap_convert_f32_bf16(const float* src, void* dst, int64_t count, void* hip_stream);

/* ------------------------------------------------------------------------
 * Step executor -- the library's runtime for one shard geometry: each packed
 * batch is planned on the host and run with one call per stage.  Not in the
 * paper; it sequences the entry points above the way a training step uses
 * them (plan before any transfer, then the shard's attention against every
 * chunk, then the backward), keeping the host cost of a step small next to
 * its kernels.
 *
 * An executor owns: a ring of 16 pinned staging buffers for the planner's lists, one
 * device list buffer, the fp32 partial outputs of the forward (grown to the
 * largest plan seen) and, with HSAP_EXEC_BACKWARD, the device doc_start
 * array and the backward's delta.  The forwards take document starts from
 * the uploaded cu_seqlens: each wave finds the document of its first query
 * by binary search and scans the boundaries among its 32 queries, so a
 * forward-only step runs no hsap_doc_start.  Buffers grow on demand; a
 * growth synchronises the stream first.
 *
 * Threading and streams: one executor is used by one host thread at a time,
 * on one device (the device current at creation), and all its calls should
 * pass the same stream: the single device list buffer is reused in stream
 * order.  Inputs and outputs are caller-owned device tensors in the layouts
 * of hsap_partial_attn_fwd_runs / hsap_partial_attn_bwd_runs.
 * --------------------------------------------------------------------- */
typedef struct hsap_executor hsap_executor;

/* Options of hsap_executor_create (bit mask). */
enum {
  HSAP_EXEC_BACKWARD = 1,  /* also plan k-major and MAJOR_Q_ALL runs, own delta */
  HSAP_EXEC_FUSED = 2      /* also plan MAJOR_Q_ALL runs for the fused forward   */
};

/* What the current plan holds (hsap_executor_info). */
typedef struct {
  int64_t num_tiles;        /* non-empty tiles over all ring steps          */
  int64_t num_full_tiles;   /* of which FULL                                 */
  int64_t useful_pairs;     /* allowed (query, key) pairs per head           */
  int64_t num_runs_q;       /* q-major runs (forward, dQ)                    */
  int64_t num_runs_k;       /* k-major runs (dK, dV); 0 without BACKWARD     */
  int64_t num_runs_all;     /* MAJOR_Q_ALL runs; 0 without FUSED or BACKWARD */
  int32_t num_parts;        /* partial outputs the forward writes and merges */
  int32_t split_length;     /* max_run_tiles used for the q-major runs (0: none) */
  int32_t chunks_with_tiles;
  int32_t final_q_tiles;    /* q-tiles whose only part the partial forward
                               writes as final output (the merge skips them) */
  uint64_t chunk_mask;      /* bit c set: chunk c has tiles (P <= 64)        */
} hsap_exec_info;

/*
 * hsap_executor_create -- an executor for the shard and heads in `desc`
 * (same supported shapes as hsap_partial_attn_fwd_runs; with HSAP_EXEC_BACKWARD
 * also those of hsap_partial_attn_bwd_runs, checked here: HSAP_ERR_UNSUPPORTED
 * before anything is allocated).
 *   options        HSAP_EXEC_* bits.
 *   max_run_tiles  q-major split: -1 picks hsap_split_length per plan from
 *                  hsap_fwd_resident_workgroups of the device current at
 *                  creation, 0 never splits, > 0 is used as given.  A plan whose split would need more than
 *                  HSAP_MAX_MERGE_PARTS partials is planned without split.
 *   out            receives the executor; NULL on failure.
 * Returns HSAP_ERR_HIP when device or pinned memory cannot be allocated.
 */
hsap_status hsap_executor_create(const hsap_attn_desc* desc, int32_t options, int32_t max_run_tiles,
                                 hsap_executor** out);

/* Waits for the device, then frees everything the executor owns.  NULL is a
 * no-op. */
void hsap_executor_destroy(hsap_executor* ex);

/*
 * hsap_executor_plan -- plan one packed batch: hsap_plan, hsap_plan_runs for
 * the q-major runs (partial slots renumbered densely 0..num_parts-1 in
 * increasing original slot order) and, per the options, the k-major and
 * MAJOR_Q_ALL runs; then one asynchronous upload of every list and
 * cu_seqlens from a pinned staging buffer, and (HSAP_EXEC_BACKWARD only)
 * hsap_doc_start, on `stream`.
 * The host blocks only when the staging buffer it is about to reuse may not
 * have been uploaded yet: it waits for an event recorded after every 8th
 * upload (events cost the stream a gap each), at most 16 plans in flight.
 *   cu_seqlens  host int32 [num_docs + 1] for the executor's N (rules of
 *               hsap_plan); read before the call returns.
 */
hsap_status hsap_executor_plan(hsap_executor* ex, const int32_t* cu_seqlens, int32_t num_docs, void* hip_stream);

/* Counts of the current plan; HSAP_ERR_INVALID_ARG before the first plan. */
hsap_status hsap_executor_info(const hsap_executor* ex, hsap_exec_info* info);

/*
 * hsap_executor_forward -- the shard's attention against every chunk for the
 * current plan.  fused = 0: hsap_partial_attn_fwd_runs over all q-major runs into
 * the executor's partials, then hsap_lse_merge of the num_parts partials --
 * except that a q-tile whose tiles all lie in one chunk, in one unsplit run,
 * has a single part: that run writes its final O (bf16) and LSE to o_out /
 * lse_out directly and the merge leaves those rows alone (the merge of one
 * part returns it unchanged, so the result is the same bit for bit).
 * fused = 1 (needs HSAP_EXEC_FUSED): hsap_attn_fwd_fused.
 *   q        device bf16 [n, Hq, d];  k, v  device bf16 [P, n, Hkv, d].
 *   o_out    device bf16 [n, Hq, d];  lse_out  device fp32 [Hq, n].
 */
hsap_status hsap_executor_forward(hsap_executor* ex, const void* q, const void* k, const void* v, int32_t fused,
                                  void* o_out, float* lse_out, void* hip_stream);

/*
 * hsap_executor_partial_forward, hsap_executor_merge -- the two stages of
 * hsap_executor_forward(fused = 0), callable one by one (e.g. to time them):
 * the partial attention of every q-major run into the executor's partials
 * (single-part q-tiles straight into o_out / lse_out), then the merge of the
 * other rows into o_out / lse_out.  The merge reads the partials of the last
 * partial forward; call them in this order, after the same plan, with the
 * same outputs.
 */
hsap_status hsap_executor_partial_forward(hsap_executor* ex, const void* q, const void* k, const void* v,
                                          void* o_out, float* lse_out, void* hip_stream);
hsap_status hsap_executor_merge(hsap_executor* ex, void* o_out, float* lse_out, void* hip_stream);

/*
 * hsap_executor_backward -- gradients of the forward for the current plan
 * (needs HSAP_EXEC_BACKWARD): zeroes the dk and dv rows of the k-tiles that
 * no query of the shard reaches in the chunks with tiles (the plan lists
 * them), then the kernels of hsap_attn_bwd_bf16 over the k-major and
 * MAJOR_Q_ALL runs, which write every other row of those chunks.  The dQ
 * kernel runs first and computes the preprocess (delta of
 * hsap_attn_bwd_preprocess) for its rows from o and d_o; the dK/dV kernel
 * reads it.
 *   q, k, v  as for the forward;  d_o, o  device bf16 [n, Hq, d] (o: the
 *            forward's output);  lse  device fp32 [Hq, n] (the forward's).
 *   dq       device bf16 [n, Hq, d].
 *   dk, dv   device bf16 [P, n, Hkv, d], sharded order: the rows of every
 *            chunk in hsap_exec_info.chunk_mask are written; the rows of a
 *            chunk without tiles are left untouched (this shard sends it no
 *            gradient: its contribution is zero).
 */
hsap_status hsap_executor_backward(hsap_executor* ex, const void* q, const void* k, const void* v, const void* d_o,
                                   const void* o, const float* lse, void* dq, void* dk, void* dv, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* HSAP_H */
