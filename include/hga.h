/*
 * hga.h - C ABI of the MI355X (gfx950) Hierarchical Global Attention hot path.
 *
 * The method (paper "Long-Context Fine-Tuning with Limited VRAM", Sec. 2.1 and
 * Fig. 1) routes each query block in two levels and then attends exact tokens:
 *   1. every closed chunk of C tokens and every group of g tokens has a key
 *      summary (the mean key);
 *   2. the block scores the chunk summaries and keeps the top_chunks best,
 *      besides fixed sink and local windows;
 *   3. it opens those chunks at group level and keeps the top_groups best;
 *   4. it runs causal softmax attention over the exact K/V of the sink window,
 *      the selected groups and the local window.
 * Routing carries no gradient; the backward (Sec. 2.1 closing paragraph and
 * Sec. 2.2) gives dQ for every query and dK/dV only to tokens of the active,
 * differentiable segment.
 *
 * Conventions shared by every entry point:
 *   - Tensor pointers are DEVICE pointers owned by the caller. The library never
 *     allocates, frees or keeps device memory; scratch space is passed in as
 *     `workspace` (size from hga_workspace_size).
 *   - Every call is asynchronous and ordered on `stream` (a hipStream_t; NULL
 *     is the default stream). No call synchronizes the device.
 *   - Argument errors are detected on the host before anything is launched and
 *     reported as HGA_ERR_INVALID_ARG / HGA_ERR_UNSUPPORTED; a failed launch is
 *     reported as HGA_ERR_HIP. No C++ exception crosses this interface.
 *   - Token-major layouts: Q/O/dO are [row][n_q_heads][head_dim], K/V are
 *     [token][n_kv_heads][head_dim]. Strides are in ELEMENTS; the head_dim axis
 *     is contiguous and every row start must be 16-byte aligned.
 *   - GQA: query head hq reads kv head hq / (n_q_heads / n_kv_heads). One
 *     routing decision is made per (query block, kv head) and is shared by the
 *     query heads of that kv head.
 *   - The library holds no state and is thread-safe; calls that share output
 *     buffers must be ordered by the caller.
 */
#ifndef HGA_H
#define HGA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { HGA_F32 = 0, HGA_BF16 = 1 } hga_dtype_t;

typedef enum {
  HGA_OK = 0,
  HGA_ERR_INVALID_ARG = -1, /* null pointer, bad range, divisibility, alignment */
  HGA_ERR_UNSUPPORTED = -2, /* valid problem outside what the library implements */
  HGA_ERR_WORKSPACE = -3,   /* workspace missing or smaller than hga_workspace_size */
  HGA_ERR_HIP = -4          /* a HIP launch or runtime call failed */
} hga_status_t;

/* Problem statement of one attention layer (Sec. 2.1; the paper's defaults are
 * 64-token chunks, 8-token groups and 8 routed chunks, Sec. 3). */
typedef struct {
  int32_t n_q_heads;     /* Hq; multiple of n_kv_heads, Hq / Hkv in {1, 2, 4, 8}      */
  int32_t n_kv_heads;    /* Hkv >= 1                                                   */
  int32_t head_dim;      /* d in {64, 128}                                             */
  int32_t chunk_size;    /* C; the library supports C == 64                            */
  int32_t group_size;    /* g; power of two dividing C                                 */
  int32_t query_block;   /* B; the library supports B == C == 64                       */
  int32_t top_chunks;    /* k_c in [0, 64]: chunks kept per (block, kv head)           */
  int32_t top_groups;    /* k_g in [0, 64]: groups kept among the kept chunks' groups  */
  int32_t sink_tokens;   /* Ws: multiple of C; tokens [0, Ws) are always attended      */
  int32_t local_tokens;  /* Wl: multiple of C, >= B; the Wl tokens ending at the block */
                         /* end (diagonal block included) are always attended          */
  float softmax_scale;   /* <= 0 selects 1/sqrt(head_dim)                              */
  hga_dtype_t dtype;     /* element type of Q, K, V, O and dO                          */
  int32_t bwd_kv_parts;  /* dK/dV work items per (active chunk, kv head) in            */
                         /* hga_attend_bwd: 0 = the library's choice (two query-head  */
                         /* subsets when the call has little routable history, which */
                         /* shortens one call), 1 = one (least total work, for       */
                         /* callers that overlap several backward calls), 2 = two    */
                         /* when Hq / Hkv >= 2; other values HGA_ERR_INVALID_ARG     */
} hga_config_t;

/* Element strides of a token-major tensor; the head_dim axis is contiguous.
 * Every call requires strides below 2^32 bytes and token positions (q_begin +
 * n_q, t_end) at most 2^31 (else HGA_ERR_INVALID_ARG): row offsets are then one
 * 32 x 32 -> 64-bit product in the kernels. */
typedef struct {
  int64_t token;
  int64_t head;
} hga_strides_t;

/*
 * hga_build_summaries - the key summaries of Sec. 2.1 items 1-2, built from
 * the same keys attention uses: the mean key of every complete group of g
 * tokens and of every complete chunk of C tokens that lies inside
 * [t_begin, t_end), computed exactly and rounded once to float32.
 *
 *   K          [t_end rows used][Hkv][d] of cfg->dtype, strides ks.
 *   t_begin    multiple of C; t_end > t_begin. Groups/chunks that end after
 *              t_end are not written (call again when they close).
 *   chunk_sum  float32 [Hkv][d/4][chunk_cap][4]: element e of chunk c's
 *              summary of kv head h at ((h * d/4 + e/4) * chunk_cap + c) * 4
 *              + e % 4, written for every chunk with c*C >= t_begin and
 *              (c+1)*C <= t_end. (Quads of consecutive chunks are adjacent,
 *              so the routing scan, one chunk per lane, reads contiguously.)
 *   group_sum  float32 [Hkv][d/4][group_cap][4]: group j likewise with g.
 *   chunk_cap, group_cap  row capacity of the two tables (>= t_end/C, t_end/g).
 * Summaries of earlier tokens are left untouched, so a caller processing a
 * long context segment by segment calls this once per segment.
 */
hga_status_t hga_build_summaries(const hga_config_t* cfg, const void* K, hga_strides_t ks,
                                 int64_t t_begin, int64_t t_end,
                                 float* chunk_sum, int64_t chunk_cap,
                                 float* group_sum, int64_t group_cap, void* stream);

/*
 * hga_route - two-level routing of Sec. 2.1 items 1-2 (Fig. 1: score, top-k,
 * top-k) for the query rows [q_begin, q_begin + n_q) held in Q.
 *
 * For each query block b and kv head h:
 *   qbar     = mean of the block's B rows over the G query heads of h;
 *   windows  : local = [max(0, end - Wl), end) with end the block end,
 *              sink  = [0, min(Ws, local start));
 *   candidates = closed chunks c with c*C >= Ws and (c+1)*C <= local start;
 *   sel_chunks = the top_chunks candidates by qbar . chunk_sum (all if fewer);
 *   sel_groups = the top_groups of all groups of sel_chunks by qbar . group_sum.
 * Scores are accumulated in float64; equal scores keep the lower index.
 *
 *   Q          rows [0, n_q) of cfg->dtype, strides qs; row r is query position q_begin + r.
 *   q_begin, n_q  multiples of B; n_q > 0.
 *   chunk_sum / group_sum  tables from hga_build_summaries covering every
 *              chunk/group that closes before q_begin + n_q.
 *   sel_chunks int32 [n_q/B][Hkv][top_chunks]: ascending chunk ids, -1 padded.
 *   sel_groups int32 [n_q/B][Hkv][top_groups]: ascending global group ids, -1 padded.
 *   n_sel_groups int32 [n_q/B][Hkv]: number of valid entries in sel_groups.
 *   workspace  device scratch of hga_workspace_size(cfg, HGA_OP_ROUTE, ...) bytes;
 *              routing needs none (size 0), and NULL is then accepted.
 * Limit: top_chunks * C / g <= 1024 candidate groups (else
 * HGA_ERR_UNSUPPORTED). The context length has none of its own (Sec. 2.2):
 * beyond 8,192 candidate chunks per block the chunks are scored and selected
 * in rounds of 512 with a running selection, which selects as the whole list.
 */
hga_status_t hga_route(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                       int64_t q_begin, int64_t n_q,
                       const float* chunk_sum, int64_t chunk_cap,
                       const float* group_sum, int64_t group_cap,
                       int32_t* sel_chunks, int32_t* sel_groups, int32_t* n_sel_groups,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * hga_attend_fwd - exact-token attention of Sec. 2.1 item 3: for query i of
 * block b and query head hq (kv head h = hq / G), softmax over the tokens t of
 * b's routed set for h (sink window, selected groups, local window) with
 * t <= i, scaled by softmax_scale, applied to the exact V rows.
 *
 *   Q          rows [0, n_q), strides qs (row r = position q_begin + r).
 *   K, V       rows [0, q_begin + n_q), strides ks / vs.
 *   sel_groups, n_sel_groups  as written by hga_route for the same rows.
 *   O          rows [0, n_q) of cfg->dtype, strides os (bf16 results are rounded to nearest even).
 *   lse        float32 [n_q][Hq]: natural-log log-sum-exp of the scaled scores.
 *   o_f32      optional (may be NULL) float32 [n_q][Hq][d], dense: O before its
 *              final rounding to cfg->dtype. When given with bf16 inputs, P
 *              also enters P.V as a pair of bf16 values (hi + lo), so this copy
 *              is accurate to ~2^-17 relative; passing it to hga_attend_bwd
 *              makes the backward's row term D = rowsum(dO * O) that accurate.
 * Accumulation is float32; with bf16 inputs P is rounded to bf16 before P.V.
 */
hga_status_t hga_attend_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                            const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                            int64_t q_begin, int64_t n_q,
                            const int32_t* sel_groups, const int32_t* n_sel_groups,
                            void* O, hga_strides_t os, float* lse, float* o_f32, void* stream);

/*
 * hga_route_attend_fwd - hga_route then hga_attend_fwd on the same query rows
 * (Sec. 2.1 items 1-3 in sequence): the arguments and results of both calls,
 * routing tables included (the backward reads them). For calls whose query
 * blocks alone do not fill the GPU (a training segment) the two run as one
 * launch: each forward workgroup routes its own block, keeping the selection
 * in LDS, and writes the routing tables on the way; the results equal those
 * of the two calls. Larger calls launch the two kernels. Same errors as the
 * two calls, checked before anything is launched.
 */
hga_status_t hga_route_attend_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                  const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                  int64_t q_begin, int64_t n_q, const float* chunk_sum,
                                  int64_t chunk_cap, const float* group_sum, int64_t group_cap,
                                  int32_t* sel_chunks, int32_t* sel_groups, int32_t* n_sel_groups,
                                  void* O, hga_strides_t os, float* lse, float* o_f32,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * hga_gather_routed - the exact-token gather of Sec. 2.1 item 3 on its own:
 * the K and V rows of every (query block, kv head)'s routed set written to
 * compact buffers, so that the gather can be measured apart from the
 * attention (hga_attend_gathered_fwd then attends over the buffers). The
 * attention entry points never materialise these rows: they gather them
 * straight into on-chip tiles.
 *
 *   K, V       rows [0, q_begin + n_q) of cfg->dtype, strides ks / vs.
 *   sel_groups, n_sel_groups  as written by hga_route for the same rows.
 *   Kc, Vc     cfg->dtype [n_q/B][Hkv][r_cap][d], dense, caller-owned. Row p
 *              of slot (b, h) holds position p of the block's routed set, in
 *              the order sink window, local window (diagonal block last),
 *              selected groups (ascending ids); rows from the set size R up
 *              to the next multiple of 64 are written as zeros, later rows
 *              are not written.
 *   r_cap      rows per slot: a multiple of 64 that is at least
 *              sink_tokens + local_tokens + top_groups * group_size rounded
 *              up to a multiple of 64 (else HGA_ERR_INVALID_ARG).
 */
hga_status_t hga_gather_routed(const hga_config_t* cfg, const void* K, hga_strides_t ks,
                               const void* V, hga_strides_t vs, int64_t q_begin, int64_t n_q,
                               const int32_t* sel_groups, const int32_t* n_sel_groups,
                               void* Kc, void* Vc, int64_t r_cap, void* stream);

/*
 * hga_attend_gathered_fwd - hga_attend_fwd (Sec. 2.1 item 3) with the routed
 * K/V rows read from the compact buffers of hga_gather_routed instead of
 * being gathered from K and V. The attention itself is the same code in the
 * same order, so O, lse and o_f32 equal those of hga_attend_fwd bit for bit.
 *
 *   Kc, Vc, r_cap  as written by hga_gather_routed for the same rows.
 *   n_sel_groups   the routing counts (the set sizes follow from them).
 *   Q, O, lse, o_f32  as for hga_attend_fwd.
 */
hga_status_t hga_attend_gathered_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                     const void* Kc, const void* Vc, int64_t r_cap,
                                     int64_t q_begin, int64_t n_q, const int32_t* n_sel_groups,
                                     void* O, hga_strides_t os, float* lse, float* o_f32,
                                     void* stream);

/*
 * hga_attend_bwd - backward of hga_attend_fwd with the routing held constant
 * (Sec. 2.1: routing runs without gradients; Sec. 2.2: only the active
 * segment is differentiable, history K/V is detached).
 *
 *   O, lse     the forward's outputs for the same inputs.
 *   o_f32      optional (may be NULL): the forward's float32 copy of O. When
 *              given, D = rowsum(dO * O) uses it; otherwise D uses O as
 *              rounded to cfg->dtype, whose error (2^-9 relative for bf16)
 *              reaches dQ multiplied by the key magnitudes.
 *   dO         upstream gradient, rows [0, n_q) of cfg->dtype, strides dos.
 *   grad_begin first token that receives dK/dV: multiple of C, <= q_begin.
 *   dQ         float32 [n_q][Hq][d], overwritten.
 *   dK, dV     float32 [q_begin + n_q - grad_begin][Hkv][d], overwritten; row r
 *              is token grad_begin + r, summed over the G query heads of each
 *              kv head. Tokens before grad_begin receive nothing.
 *   workspace  device scratch of hga_workspace_size(cfg, HGA_OP_BWD, ...) bytes
 *              (never 0): D of every (query row, query head), n_q * Hq
 *              floats rounded up to 256 bytes, then, when the call starts
 *              with little routable history (fewer than 6 * top_chunks
 *              candidate chunks before its first block), the partial dK/dV
 *              sums of 2 subsets of the query heads: most routed keys then
 *              lie in the active segment and the dK/dV work of each chunk is
 *              split over those subsets. Its contents need no
 *              initialisation.
 * A first kernel forms D = rowsum(dO * O) of every row; one launch then
 * computes dQ (query-major) and dK/dV (key-major) side by side. dK/dV are
 * accumulated in fixed order (no atomics; the split partials are summed in a
 * fixed order by a third kernel): results are bitwise reproducible run to
 * run. With bf16 inputs dS enters dQ = dS K as a pair of bf16 values
 * (hi + lo), since dQ scales dS by raw key magnitudes.
 */
hga_status_t hga_attend_bwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                            const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                            const void* O, hga_strides_t os, const float* o_f32,
                            const void* dO, hga_strides_t dos,
                            const float* lse, int64_t q_begin, int64_t n_q, int64_t grad_begin,
                            const int32_t* sel_groups, const int32_t* n_sel_groups,
                            float* dQ, float* dK, float* dV,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * hga_route_rows - two-level routing with one decision per query row instead
 * of per block: routing at generation time, a decode step being one row
 * (Sec. 1, last result, and Sec. 7: routed generation), and over a whole
 * training segment a strictly causal variant of the method (Sec. 6.1: a
 * routing decision shared by a block lets an early query's attended set
 * depend on later queries of the block).
 *
 * For each query row i (position q_begin + i) and kv head h:
 *   qbar     = mean of row i's G query-head rows of kv head h;
 *   windows and candidate chunks: those of the B-block holding the row
 *              (as in hga_route), so rows of one block share them;
 *   sel_chunks / sel_groups: as in hga_route, ranked with the row's qbar.
 * Scores are accumulated in float64; equal scores keep the lower index.
 *
 *   Q          rows [0, n_q) of cfg->dtype, strides qs; row i is position q_begin + i.
 *   q_begin    any position >= 0; n_q >= 1 (any count).
 *   chunk_sum / group_sum  as for hga_route: every chunk closed before the
 *              local window of the last row's block must be summarised.
 *   sel_chunks int32 [n_q][Hkv][top_chunks], sel_groups int32
 *              [n_q][Hkv][top_groups] (ascending, -1 padded), n_sel_groups
 *              int32 [n_q][Hkv].
 * Needs no workspace. Limit: top_chunks * C / g <= 1024 (else
 * HGA_ERR_UNSUPPORTED); a row's candidate chunks are scored and selected in
 * rounds of 4,096 with a running selection, so the context length has no
 * limit of its own.
 */
hga_status_t hga_route_rows(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                            int64_t q_begin, int64_t n_q,
                            const float* chunk_sum, int64_t chunk_cap,
                            const float* group_sum, int64_t group_cap,
                            int32_t* sel_chunks, int32_t* sel_groups, int32_t* n_sel_groups,
                            void* stream);

/*
 * hga_attend_rows_fwd - exact-token attention (Sec. 2.1 item 3) of each query
 * row over its own routed set from hga_route_rows: the sink window of its
 * block, its selected groups, and its block's local window up to and
 * including the row's position. Keys after the row are never read.
 *
 *   Q          rows [0, n_q), strides qs (row i = position q_begin + i).
 *   K, V       rows [0, q_begin + n_q), strides ks / vs.
 *   sel_groups, n_sel_groups  as written by hga_route_rows for the same rows.
 *   O          rows [0, n_q) of cfg->dtype, strides os (bf16 rounded to nearest even).
 *   lse        float32 [n_q][Hq], natural log.
 *   o_f32      optional (may be NULL) float32 [n_q][Hq][d], dense: O before
 *              its rounding to cfg->dtype, for hga_attend_rows_bwd.
 * Scores, softmax and accumulation in float32. With bf16 inputs P is rounded
 * to bf16 before P.V (as in hga_attend_fwd); with float32 inputs it is not.
 */
hga_status_t hga_attend_rows_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                 const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                 int64_t q_begin, int64_t n_q,
                                 const int32_t* sel_groups, const int32_t* n_sel_groups,
                                 void* O, hga_strides_t os, float* lse, float* o_f32, void* stream);

/*
 * hga_attend_rows_bwd - backward of hga_attend_rows_fwd with the routing held
 * constant (Sec. 2.1 closing paragraph; Sec. 2.2: dK/dV only for the active
 * segment): the training side of the strictly causal variant.
 *
 *   O, lse, o_f32  the forward's outputs (o_f32 optional: D = rowsum(dO * O)
 *              then uses the float32 O instead of O rounded to cfg->dtype).
 *   dO         rows [0, n_q) of cfg->dtype, strides dos.
 *   q_begin, n_q  any position >= 0; 1 <= n_q <= 4096 (else HGA_ERR_UNSUPPORTED).
 *   grad_begin multiple of C, <= q_begin: tokens [grad_begin, q_begin + n_q)
 *              receive dK/dV; earlier tokens receive nothing.
 *   dQ         float32 [n_q][Hq][d], overwritten.
 *   dK, dV     float32 [q_begin + n_q - grad_begin][Hkv][d], overwritten,
 *              summed over the G query heads of each kv head.
 *   workspace  device scratch of hga_rows_workspace_size(cfg, n_q) bytes (D
 *              of every (row, query head)); needs no initialisation.
 * Accumulation is float32. With bf16 inputs the products run on bf16
 * operands, with P and dS carried as bf16 hi + lo pairs (each enters to
 * about 2^-17 relative). dK/dV are accumulated key-major in row order with
 * no atomics: results are bitwise reproducible.
 */
hga_status_t hga_attend_rows_bwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                 const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                 const void* O, hga_strides_t os, const float* o_f32,
                                 const void* dO, hga_strides_t dos,
                                 const float* lse, int64_t q_begin, int64_t n_q, int64_t grad_begin,
                                 const int32_t* sel_groups, const int32_t* n_sel_groups,
                                 float* dQ, float* dK, float* dV,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of device workspace hga_attend_rows_bwd needs for n_q rows; 0 for an
 * invalid configuration or count. */
size_t hga_rows_workspace_size(const hga_config_t* cfg, int64_t n_q);

/*
 * Tiered storage (Sec. 2.2, Fig. 2; Sec. 2.1 item 2). The history's exact
 * K/V and the full table of group summaries may live in host RAM; device
 * memory then holds the active segment, every chunk summary, a bounded cache
 * of group summaries and the routed working set of the current call. One
 * call of a segment runs:
 *   hga_build_summaries       (group_sum may be the host table's device view)
 *   hga_route_cached          routing; group summaries from the cache when
 *                             resident, else from the host table; hit flags
 *   hga_group_cache_update    the call's missed chunks brought into the cache
 *   hga_gather_tiered         the routed exact K/V rows, history rows from
 *                             host RAM, into a compact device working set
 *   hga_attend_gathered_fwd   the forward over the working set
 *   hga_attend_gathered_bwd   the backward: dQ from the working set, dK/dV
 *                             for the active tokens from device rows
 * Every result equals that of the same calls on device-resident tensors.
 */

/* Device-mapped address of pinned host memory (hipHostMalloc, or a pinned
 * torch tensor), usable by the kernels of this library; NULL if the pointer
 * is not pinned host memory. */
void* hga_host_device_view(const void* host_ptr);

/* A bounded device cache of group summaries, a whole chunk per slot (its C/g
 * group summaries). Caller-owned device buffers:
 *   slot_of     int32 [Hkv][chunk_cap]: the slot holding each chunk, -1 if none;
 *   slot_chunk  int32 [Hkv][n_slots]: the chunk each slot holds, -1 if empty;
 *   cursor      int32 [Hkv]: the next slot to fill;
 *   groups      float32 [Hkv][d/4][n_slots * C/g][4], quad-major like group_sum.
 * n_slots in [1, 4096]; chunk_cap in [1, 262144] and equal to the chunk_cap
 * passed with the chunk summaries. Replacement is first in, first out: the
 * chunks a call chose that were not resident enter in ascending chunk order
 * (the last n_slots of them when more), so the cache's contents depend only on
 * the sequence of routing calls. */
typedef struct {
  int32_t* slot_of;
  int32_t* slot_chunk;
  int32_t* cursor;
  float* groups;
  int64_t n_slots;
  int64_t chunk_cap;
} hga_group_cache_t;

/* Empties the cache (no slot holds a chunk, cursor 0). */
hga_status_t hga_group_cache_clear(const hga_config_t* cfg, const hga_group_cache_t* cache, void* stream);

/*
 * hga_route_cached - hga_route with the group summaries of the chosen chunks
 * read from the cache where resident and from group_sum (the full table,
 * e.g. the device view of a host table) otherwise; the routing is the same.
 *   cache_hit  int32 [n_q/B][Hkv][top_chunks]: 1 where the chosen chunk of that
 *              rank (sel_chunks) was resident when the call began, else 0;
 *              entries past the chosen count are not written.
 * The cache is only read: hga_group_cache_update brings the misses in.
 */
hga_status_t hga_route_cached(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                              int64_t q_begin, int64_t n_q,
                              const float* chunk_sum, int64_t chunk_cap,
                              const float* group_sum, int64_t group_cap,
                              const hga_group_cache_t* cache,
                              int32_t* sel_chunks, int32_t* sel_groups, int32_t* n_sel_groups,
                              int32_t* cache_hit, void* workspace, size_t workspace_bytes, void* stream);

/* Brings the chunks that a hga_route_cached call over the same rows chose and
 * missed into the cache (group summaries copied from group_sum). */
hga_status_t hga_group_cache_update(const hga_config_t* cfg, const hga_group_cache_t* cache,
                                    const float* group_sum, int64_t group_cap,
                                    int64_t q_begin, int64_t n_q,
                                    const int32_t* sel_chunks, const int32_t* cache_hit, void* stream);

/*
 * hga_gather_tiered - hga_gather_routed over K/V split in two tiers: tokens
 * [0, hist_end) from K_hist / V_hist (strides hs; host RAM through its device
 * view, or device memory), tokens [hist_end, q_begin + n_q) from K_act /
 * V_act (strides as; row 0 is token hist_end). hist_end is a multiple of C,
 * <= q_begin. Kc, Vc, r_cap and the row order as for hga_gather_routed.
 */
hga_status_t hga_gather_tiered(const hga_config_t* cfg, const void* K_hist, const void* V_hist,
                               hga_strides_t hs, int64_t hist_end,
                               const void* K_act, const void* V_act, hga_strides_t as,
                               int64_t q_begin, int64_t n_q,
                               const int32_t* sel_groups, const int32_t* n_sel_groups,
                               void* Kc, void* Vc, int64_t r_cap, void* stream);

/*
 * hga_attend_gathered_bwd - hga_attend_bwd with the routed K/V rows read
 * from the compact working set (Kc, Vc, r_cap as written by hga_gather_routed
 * or hga_gather_tiered) for dQ, and the keys that receive dK/dV read from
 * K_act / V_act, device rows [act_begin, q_begin + n_q) (row 0 = token
 * act_begin; act_begin a multiple of C, <= grad_begin). Other arguments,
 * the workspace and the results as for hga_attend_bwd (bit for bit).
 */
hga_status_t hga_attend_gathered_bwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                     const void* Kc, const void* Vc, int64_t r_cap,
                                     const void* K_act, const void* V_act, hga_strides_t as,
                                     int64_t act_begin,
                                     const void* O, hga_strides_t os, const float* o_f32,
                                     const void* dO, hga_strides_t dos, const float* lse,
                                     int64_t q_begin, int64_t n_q, int64_t grad_begin,
                                     const int32_t* sel_groups, const int32_t* n_sel_groups,
                                     float* dQ, float* dK, float* dV,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * hga_attend_bwd_noalloc - hga_attend_bwd for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same computation and results, with the
 * backward's workspace taken from a static buffer of the library instead of
 * an argument. No device memory is allocated or freed by the call.
 *
 *   Arguments as for hga_attend_bwd, without workspace / workspace_bytes.
 *   Limit: calls whose hga_workspace_size(cfg, HGA_OP_BWD, ...) exceeds
 *          HGA_NOALLOC_SCRATCH_BYTES (48 MiB) return HGA_ERR_WORKSPACE before
 *          anything is launched.
 *   The buffer is one per device, held from the first call on that device
 *   until the process ends, and shared by every call on that device: calls
 *   that overlap on one device (other streams, other threads) race on it and
 *   must be ordered by the caller. Each call rewrites what it reads; nothing
 *   needs clearing between calls.
 */
#define HGA_NOALLOC_SCRATCH_BYTES (48u << 20)
hga_status_t hga_attend_bwd_noalloc(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                    const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                    const void* O, hga_strides_t os, const float* o_f32,
                                    const void* dO, hga_strides_t dos,
                                    const float* lse, int64_t q_begin, int64_t n_q, int64_t grad_begin,
                                    const int32_t* sel_groups, const int32_t* n_sel_groups,
                                    float* dQ, float* dK, float* dV, void* stream);

enum { HGA_OP_ROUTE = 0, HGA_OP_BWD = 1 };

/* Bytes of device workspace hga_route (op HGA_OP_ROUTE) or hga_attend_bwd
 * (op HGA_OP_BWD) needs for the query rows [q_begin, q_begin + n_q) and, for
 * the backward, gradients from grad_begin on (ignored for HGA_OP_ROUTE);
 * 0 for an invalid configuration or range. */
size_t hga_workspace_size(const hga_config_t* cfg, int op, int64_t q_begin, int64_t n_q,
                          int64_t grad_begin);

/* Static, NUL-terminated description of a status code. */
const char* hga_status_string(hga_status_t status);

#ifdef __cplusplus
}
#endif
#endif /* HGA_H */
