// Internal launch interface between the C ABI layer (api.hip) and the kernels.
// Everything here is validated by the ABI layer before a launcher is called.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hga {

struct SummaryArgs {
  const void* K;
  int64_t k_tok, k_head;
  int64_t t_begin, t_end;
  float* chunk_sum;
  int64_t chunk_cap;
  float* group_sum;
  int64_t group_cap;
  int n_kv_heads, head_dim, group_shift;
};

struct RouteArgs {
  const void* Q;            // query rows [n_qb * 64][Hq][D]
  int64_t q_tok, q_head;
  int gqa;
  const float* chunk_sum;   // [Hkv][chunk_cap][D]
  int64_t chunk_cap;
  const float* group_sum;   // [Hkv][group_cap][D]
  int64_t group_cap;
  int32_t* sel_chunks;      // [n_qb][Hkv][k_c]
  int32_t* sel_groups;      // [n_qb][Hkv][k_g]
  int32_t* n_sel;           // [n_qb][Hkv]
  int64_t q_begin;
  int n_qb, n_kv_heads;
  int top_chunks, top_groups, group_shift;
  int sink_tokens, local_tokens;
  int first_cand;           // ceil(Ws / C)
  int score_stride;         // doubles of LDS per block for scores
  int round_rows;           // > 0 (TB > 1 only): candidates are scored and selected in rounds of this many rows
  // optional group-summary cache (null: every group row from group_sum)
  const int32_t* slot_of;   // [Hkv][chunk_cap]: cache slot holding the chunk's groups, -1 if none
  const float* gcache;      // [Hkv][D/4][gcache_cap][4]: cached group summaries
  int64_t gcache_cap;       // rows of gcache per head (slots * groups per chunk)
  int32_t* cache_hit;       // [n_qb][Hkv][k_c]: 1 if the chosen chunk was resident, else 0
};

__device__ inline void prefetch_args(const RouteArgs& a) {
  asm volatile("" ::"s"(a.Q), "s"(a.sel_chunks), "s"(a.slot_of));
}

struct AttnArgs {
  const void* Q;
  int64_t q_tok, q_head;
  const void* K;
  int64_t k_tok, k_head;
  const void* V;
  int64_t v_tok, v_head;
  const void* O;            // forward output (backward input)
  int64_t o_tok, o_head;
  void* Out;                // forward: O; unused by backward
  int64_t out_tok, out_head;
  const void* dO;
  int64_t do_tok, do_head;
  float* lse;               // forward writes, backward reads
  float* o32;               // optional float32 O [n_q][Hq][D]: forward writes, backward reads
  const int32_t* sel_groups;
  const int32_t* n_sel;
  float* dQ;
  float* dK;
  float* dV;
  int64_t q_begin, grad_begin;
  int n_qb, n_q_heads, n_kv_heads, gqa;
  int top_groups, group_shift;
  int sink_tokens, local_tokens;
  int n_act_chunks;
  float* dvec;              // backward: rowsum(dO * O) [n_q][Hq], from the row-dot kernel
  int kv_parts;             // dK/dV work items per (chunk, kv head): query-head subsets
  float* part_out;          // kv_parts > 1: partial dK then dV, [part][chunk][Hkv][64][D] each
  int64_t r_cap;            // > 0: K/V are compact routed rows [n_qb][Hkv][r_cap][D] (gather / gathered forward)
  int heavy_last;           // the forward's later blocks carry much more work: start them first
  const void* Kact;         // backward dK/dV role: the rows of the active tokens, row 0 = token act_begin
  const void* Vact;         // (a.K / a.V and act_begin 0 except over compact routed rows)
  int64_t ka_tok, ka_head, va_tok, va_head, act_begin;
  float scale, scale_log2;
};

// The kernel-argument lines a kernel reads, requested at its start: fields
// are otherwise loaded where first used, after the first barrier or branch,
// and each line that misses the scalar cache then costs a round trip on the
// kernel's critical path (one field per 64-byte line of the struct).
__device__ inline void prefetch_args(const AttnArgs& a) {
  asm volatile("" ::"s"(a.Q), "s"(a.O), "s"(a.lse), "s"(a.q_begin), "s"(a.dvec), "s"(a.scale));
}

// A bounded device cache of group summaries, whole chunks at a time (the
// C/g groups of a chunk share a slot), and the call whose misses update it.
constexpr int kMaxCacheSlots = 4096;
struct CacheArgs {
  int32_t* slot_of;          // [Hkv][chunk_cap]: slot holding the chunk's groups, -1 if none
  int32_t* slot_chunk;       // [Hkv][n_slots]: chunk held by the slot, -1 if empty
  int32_t* cursor;           // [Hkv]: next slot to fill (first in, first out)
  float* groups;             // [Hkv][D/4][n_slots * C/g][4]: the cached group summaries
  int64_t n_slots, chunk_cap;
  const float* group_sum;    // the full group-summary table (host memory, device-mapped)
  int64_t group_cap;
  const int32_t* sel_chunks; // the call's routing [n_qb][Hkv][k_c] and its hit flags
  const int32_t* cache_hit;
  int n_qb, n_kv_heads, top_chunks, gpc_shift;
};

// K and V split in two tiers: rows [0, hist_end) in host memory (device-
// mapped), rows [hist_end, ...) in device memory with row 0 = token hist_end.
struct TierArgs {
  const void* K_hist;
  const void* V_hist;
  int64_t h_tok, h_head;
  const void* K_act;
  const void* V_act;
  int64_t a_tok, a_head;
  int64_t hist_end;
};

// Summary tables, float32 [Hkv][d/4][cap][4]: float offset of quad q (elements
// 4q..4q+3) of row r of kv head h.
__host__ __device__ inline int64_t quad_off(int h, int q, int64_t r, int d, int64_t cap) {
  return (((int64_t)h * (d / 4) + q) * cap + r) * 4;
}

// Launchers return hipSuccess or the launch error. `bf16` selects the element
// type (else fp32); `d` is 64 or 128.
hipError_t launch_summaries(const SummaryArgs& a, bool bf16, hipStream_t s);
size_t route_lds_bytes(int blocks_per_wg, int score_stride, bool bf16);
hipError_t launch_route(const RouteArgs& a, bool bf16, int head_dim, int blocks_per_wg,
                        hipStream_t s);
hipError_t launch_attend_fwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s);
// Routing + forward in one launch: for calls the routing kernel would serve
// with one block per workgroup and the forward with two-head workgroups;
// route_lds is the routing's dynamic LDS for one block.
bool route_attend_fusable(const AttnArgs& a, size_t route_lds);
hipError_t launch_route_attend(const RouteArgs& ra, const AttnArgs& a, bool bf16, int head_dim,
                               size_t route_lds, hipStream_t s);
hipError_t launch_attend_bwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s);
// The routed rows of every (block, kv head) into a.K / a.V's compact copies
// kc / vc ([n_qb][Hkv][a.r_cap][D]); the forward over such copies.
hipError_t launch_gather(const AttnArgs& a, void* kc, void* vc, bool bf16, int head_dim, hipStream_t s);
hipError_t launch_attend_gathered_fwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s);

// Per-query routing and attention (rows [q_begin, q_begin + n_rows), any
// q_begin and n_rows >= 1): routing tables and set sizes are indexed by row
// instead of block. n_cand_max: the longest candidate list of the call;
// group_cand: groups of k_c chunks.
hipError_t launch_route_rows(const RouteArgs& a, int64_t n_rows, int n_cand_max, int group_cand, bool bf16,
                             int head_dim, hipStream_t s);
hipError_t launch_attend_rows_fwd(const AttnArgs& a, int64_t n_rows, bool bf16, int head_dim, hipStream_t s);
// Backward of the per-query attention: D into a.dvec, then dQ (query-major)
// and dK/dV (key-major, one workgroup per 64-token chunk of the active
// tokens and kv head; at most 4,096 rows per call).
hipError_t launch_cache_clear(const CacheArgs& c, hipStream_t s);
hipError_t launch_cache_update(const CacheArgs& c, int head_dim, hipStream_t s);
size_t cache_update_lds_bytes(int64_t chunk_cap);
// The routed rows of every (block, kv head) from the two tiers into compact
// rows kc / vc ([n_qb][Hkv][a.r_cap][D]).
hipError_t launch_tier_gather(const AttnArgs& a, const TierArgs& t, void* kc, void* vc, bool bf16, int head_dim,
                              hipStream_t s);
// The backward over compact routed rows (a.K / a.V with a.r_cap): dQ from
// them, dK/dV from a.Kact / a.Vact (device rows from token a.act_begin).
hipError_t launch_attend_gathered_bwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s);
constexpr int kRowsBwdMaxRows = 4096;
constexpr int kRowsDkvKeys = 16;  // keys per workgroup of the per-query dK/dV kernel
constexpr int kRowsRouteRound = 4096;  // candidate chunks a one-row routing workgroup scores per round
hipError_t launch_attend_rows_bwd(const AttnArgs& a, int64_t n_rows, bool bf16, int head_dim, hipStream_t s);

}  // namespace hga
