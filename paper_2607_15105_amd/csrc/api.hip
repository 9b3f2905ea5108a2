// C ABI of the HGA hot path (declared in include/hga.h): argument validation,
// workspace sizing and kernel launches on the caller's stream. Nothing here
// allocates device memory or synchronizes; every check runs on the host before
// the first launch, so invalid calls return without touching the GPU.
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "../../include/hga.h"
#include "hga_kernels.h"

namespace {

using hga::AttnArgs;

constexpr int kChunk = 64;
constexpr int kMaxGroupCand = 1024;
constexpr int64_t kMaxCacheChunks = 262144;  // chunks a group-summary cache's slot map covers

int log2_exact(int x) {
  int s = 0;
  while ((1 << s) < x) ++s;
  return (1 << s) == x ? s : -1;
}

int elem_bytes(const hga_config_t* c) { return c->dtype == HGA_BF16 ? 2 : 4; }

hga_status_t check_cfg(const hga_config_t* c) {
  if (!c) return HGA_ERR_INVALID_ARG;
  if (c->dtype != HGA_F32 && c->dtype != HGA_BF16) return HGA_ERR_INVALID_ARG;
  if (c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->n_q_heads % c->n_kv_heads != 0)
    return HGA_ERR_INVALID_ARG;
  const int G = c->n_q_heads / c->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return HGA_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return HGA_ERR_UNSUPPORTED;
  if (c->dtype == HGA_F32 && c->head_dim != 64) return HGA_ERR_UNSUPPORTED;
  if (c->chunk_size <= 0 || c->query_block <= 0) return HGA_ERR_INVALID_ARG;
  if (c->chunk_size != kChunk || c->query_block != kChunk) return HGA_ERR_UNSUPPORTED;
  if (c->group_size <= 0 || c->chunk_size % c->group_size != 0) return HGA_ERR_INVALID_ARG;
  if (log2_exact(c->group_size) < 0) return HGA_ERR_UNSUPPORTED;
  if (c->top_chunks < 0 || c->top_groups < 0) return HGA_ERR_INVALID_ARG;
  if (c->top_chunks > 64 || c->top_groups > 64) return HGA_ERR_UNSUPPORTED;
  if (c->sink_tokens < 0 || c->sink_tokens % c->chunk_size != 0) return HGA_ERR_INVALID_ARG;
  if (c->local_tokens < c->query_block || c->local_tokens % c->chunk_size != 0)
    return HGA_ERR_INVALID_ARG;
  if (!(c->softmax_scale == c->softmax_scale)) return HGA_ERR_INVALID_ARG;  // NaN
  if (c->bwd_kv_parts < 0 || c->bwd_kv_parts > 2) return HGA_ERR_INVALID_ARG;
  return HGA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Token positions stay below 2^31 and token / head strides below 4 GB, so a
// row's byte offset is one 32 x 32 -> 64-bit product in the kernels.
constexpr int64_t kMaxTokens = (int64_t)1 << 31;
constexpr int64_t kMaxStrideBytes = (int64_t)1 << 32;

hga_status_t check_tensor(const void* p, hga_strides_t s, int eb) {
  if (!p || !aligned16(p)) return HGA_ERR_INVALID_ARG;
  if (s.token <= 0 || s.head <= 0) return HGA_ERR_INVALID_ARG;
  if (s.token * eb >= kMaxStrideBytes || s.head * eb >= kMaxStrideBytes) return HGA_ERR_INVALID_ARG;
  if ((s.token * eb) % 16 != 0 || (s.head * eb) % 16 != 0) return HGA_ERR_INVALID_ARG;
  return HGA_OK;
}

hga_status_t check_rows(int64_t q_begin, int64_t n_q) {
  if (q_begin < 0 || n_q <= 0 || q_begin % kChunk != 0 || n_q % kChunk != 0)
    return HGA_ERR_INVALID_ARG;
  if (q_begin + n_q > kMaxTokens) return HGA_ERR_INVALID_ARG;
  return HGA_OK;
}

// Rows of a per-query call: any first position, at least one row.
hga_status_t check_row_range(int64_t q_begin, int64_t n_q) {
  if (q_begin < 0 || n_q <= 0 || q_begin + n_q > kMaxTokens) return HGA_ERR_INVALID_ARG;
  return HGA_OK;
}

// Routing keeps everything it needs in LDS: no workspace.
size_t route_ws(const hga_config_t* c, int64_t n_q) {
  (void)c;
  (void)n_q;
  return 0;
}
// dK/dV work items per (active chunk, kv head). Each item visits the query
// blocks that attend the chunk for a subset of the G query heads. When the
// call starts with little routable history, most routed keys fall inside the
// active segment and the key-major work grows several-fold (and concentrates
// on the early chunks), so it is split over two head subsets whose partials a
// second kernel sums. (1,024-token segments of the 16K step: two subsets
// win below 6 k_c history chunks, one above; four never won.)
int bwd_parts(const hga_config_t* c, int64_t q_begin) {
  const int G = c->n_q_heads / c->n_kv_heads;
  if (c->bwd_kv_parts == 1) return 1;
  if (c->bwd_kv_parts == 2) return G >= 2 ? 2 : 1;
  const int64_t ls = q_begin + kChunk - c->local_tokens;  // first block's local start
  const int64_t first = (c->sink_tokens + kChunk - 1) / kChunk;
  const int64_t h0 = ls > 0 && ls / kChunk > first ? ls / kChunk - first : 0;  // history candidates
  const int64_t kc = c->top_chunks > 0 ? c->top_chunks : 1;
  return h0 < 6 * kc && G >= 2 ? 2 : 1;
}

// Backward workspace: D = rowsum(dO * O) of every (query row, query head),
// then the dK and dV partials when the work is split.
size_t bwd_dvec_bytes(const hga_config_t* c, int64_t n_q) {
  return ((size_t)n_q * c->n_q_heads * sizeof(float) + 255) / 256 * 256;
}
size_t bwd_ws(const hga_config_t* c, int64_t q_begin, int64_t n_q, int64_t grad_begin) {
  const int p = bwd_parts(c, q_begin);
  const int64_t rows = q_begin + n_q - grad_begin;
  const size_t parts = p == 1 ? 0 : (size_t)2 * p * rows * c->n_kv_heads * c->head_dim * sizeof(float);
  return bwd_dvec_bytes(c, n_q) + parts;
}

float eff_scale(const hga_config_t* c) {
  return c->softmax_scale > 0.0f ? c->softmax_scale : 1.0f / sqrtf((float)c->head_dim);
}

#define HGA_TRY(expr)                       \
  do {                                      \
    const hga_status_t st_ = (expr);        \
    if (st_ != HGA_OK) return st_;          \
  } while (0)

AttnArgs attn_args(const hga_config_t* c, const void* Q, hga_strides_t qs, const void* K,
                   hga_strides_t ks, const void* V, hga_strides_t vs, int64_t q_begin, int64_t n_q,
                   const int32_t* sel_groups, const int32_t* n_sel) {
  AttnArgs a = {};
  a.Q = Q; a.q_tok = qs.token; a.q_head = qs.head;
  a.K = K; a.k_tok = ks.token; a.k_head = ks.head;
  a.V = V; a.v_tok = vs.token; a.v_head = vs.head;
  a.sel_groups = sel_groups; a.n_sel = n_sel;
  a.q_begin = q_begin;
  a.n_qb = (int)(n_q / kChunk);
  a.n_q_heads = c->n_q_heads; a.n_kv_heads = c->n_kv_heads; a.gqa = c->n_q_heads / c->n_kv_heads;
  a.top_groups = c->top_groups; a.group_shift = log2_exact(c->group_size);
  a.sink_tokens = c->sink_tokens; a.local_tokens = c->local_tokens;
  // the sink window dominates the routed set once it is several times the
  // rest of it: the set then grows with the block's position
  const int64_t fixed = (int64_t)c->local_tokens + (int64_t)c->top_groups * c->group_size;
  a.heavy_last = (int64_t)c->sink_tokens >= 4 * fixed && q_begin + n_q > 4 * fixed;
  a.scale = eff_scale(c);
  a.scale_log2 = a.scale * 1.4426950408889634f;
  return a;
}

// Validates a routing call and fills its launch arguments and the number of
// query blocks per routing workgroup.
hga_status_t route_args(const hga_config_t* cfg, const void* Q, hga_strides_t qs, int64_t q_begin,
                        int64_t n_q, const float* chunk_sum, int64_t chunk_cap, const float* group_sum,
                        int64_t group_cap, int32_t* sel_chunks, int32_t* sel_groups, int32_t* n_sel_groups,
                        void* workspace, size_t workspace_bytes, hga::RouteArgs* out, int* out_tb) {
  HGA_TRY(check_cfg(cfg));
  HGA_TRY(check_tensor(Q, qs, elem_bytes(cfg)));
  HGA_TRY(check_rows(q_begin, n_q));
  const int64_t q_end = q_begin + n_q;
  if (!chunk_sum || !group_sum || !aligned16(chunk_sum) || !aligned16(group_sum))
    return HGA_ERR_INVALID_ARG;
  if (chunk_cap < q_end / kChunk || group_cap < q_end / cfg->group_size) return HGA_ERR_INVALID_ARG;
  if (!n_sel_groups || (cfg->top_chunks > 0 && !sel_chunks) || (cfg->top_groups > 0 && !sel_groups))
    return HGA_ERR_INVALID_ARG;
  const int gshift = log2_exact(cfg->group_size);
  const int gcand = cfg->top_chunks << (6 - gshift);
  if (gcand > kMaxGroupCand) return HGA_ERR_UNSUPPORTED;
  const size_t need = route_ws(cfg, n_q);
  if (need > 0 && (!workspace || workspace_bytes < need || !aligned16(workspace)))
    return HGA_ERR_WORKSPACE;

  const int n_qb = (int)(n_q / kChunk);
  const int first_cand = (cfg->sink_tokens + kChunk - 1) / kChunk;
  const int64_t last_ls = q_end - cfg->local_tokens > 0 ? q_end - cfg->local_tokens : 0;
  const int n_cand_max = (int)(last_ls / kChunk - first_cand > 0 ? last_ls / kChunk - first_cand : 0);
  int stride = n_cand_max > gcand ? n_cand_max : gcand;  // score slots per block
  if (stride < 1) stride = 1;
  const bool bf16 = cfg->dtype == HGA_BF16;
  // One block per workgroup while the (block, kv head) pairs fit the chip's
  // 256 CUs: that kernel gives its registers to latency and runs one
  // workgroup per CU. Beyond that, several blocks per workgroup share each
  // chunk-summary row read (three workgroups per CU): two blocks, or four
  // from 4,096 pairs with long candidate lists. Four blocks always score and
  // select in rounds of 512 rows, so the score table stays small enough for
  // three workgroups per CU (a whole list of 2,043 candidates at 131K took
  // 64 KB: one workgroup per CU). Measured, whole job: 131K 0.53 ms (four,
  // rounds) against 0.59 (two); 64K 0.236 against 0.254; 32K, with at most
  // 507 candidates, two blocks 0.124 against 0.127 (four).
  const int64_t pairs = (int64_t)n_qb * cfg->n_kv_heads;
  int tb = 1, round_rows = 0;
  if (pairs > 256) {
    tb = pairs >= 4096 && n_cand_max > 768 ? 4 : 2;
    if (tb == 4 || hga::route_lds_bytes(2, stride, bf16) > 65536) {
      round_rows = 512;
      stride = 64 + round_rows > gcand ? 64 + round_rows : gcand;
    }
  }
  // One block per workgroup keeps its whole candidate list in LDS (up to
  // 8,192 chunks); a longer list is scored and selected in rounds, which the
  // several-block kernel does, so the context length has no limit of its own.
  if (tb == 1 && hga::route_lds_bytes(1, stride, bf16) > 65536) {
    tb = 2;
    round_rows = 512;
    stride = 64 + round_rows > gcand ? 64 + round_rows : gcand;
  }
  if (hga::route_lds_bytes(tb, stride, bf16) > 65536) return HGA_ERR_UNSUPPORTED;

  hga::RouteArgs ra = {};
  ra.Q = Q; ra.q_tok = qs.token; ra.q_head = qs.head;
  ra.gqa = cfg->n_q_heads / cfg->n_kv_heads;
  ra.chunk_sum = chunk_sum; ra.chunk_cap = chunk_cap;
  ra.group_sum = group_sum; ra.group_cap = group_cap;
  ra.sel_chunks = sel_chunks; ra.sel_groups = sel_groups; ra.n_sel = n_sel_groups;
  ra.q_begin = q_begin; ra.n_qb = n_qb; ra.n_kv_heads = cfg->n_kv_heads;
  ra.top_chunks = cfg->top_chunks; ra.top_groups = cfg->top_groups; ra.group_shift = gshift;
  ra.sink_tokens = cfg->sink_tokens; ra.local_tokens = cfg->local_tokens;
  ra.first_cand = first_cand; ra.score_stride = stride; ra.round_rows = round_rows;
  *out = ra;
  *out_tb = tb;
  return HGA_OK;
}

// Validates a forward call and fills its launch arguments.
hga_status_t fwd_args(const hga_config_t* cfg, const void* Q, hga_strides_t qs, const void* K,
                      hga_strides_t ks, const void* V, hga_strides_t vs, int64_t q_begin, int64_t n_q,
                      const int32_t* sel_groups, const int32_t* n_sel_groups, void* O, hga_strides_t os,
                      float* lse, float* o_f32, AttnArgs* out) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_tensor(Q, qs, eb));
  HGA_TRY(check_tensor(K, ks, eb));
  HGA_TRY(check_tensor(V, vs, eb));
  HGA_TRY(check_tensor(O, os, eb));
  HGA_TRY(check_rows(q_begin, n_q));
  if (!lse || !n_sel_groups || (cfg->top_groups > 0 && !sel_groups)) return HGA_ERR_INVALID_ARG;
  if (o_f32 && !aligned16(o_f32)) return HGA_ERR_INVALID_ARG;
  AttnArgs a = attn_args(cfg, Q, qs, K, ks, V, vs, q_begin, n_q, sel_groups, n_sel_groups);
  a.Out = O; a.out_tok = os.token; a.out_head = os.head;
  a.lse = lse;
  a.o32 = o_f32;
  *out = a;
  return HGA_OK;
}

}  // namespace

// Scratch of hga_attend_bwd_noalloc: the backward's workspace (D of every
// row, then the split dK/dV partials) for callers that cannot allocate. Each
// device that runs the entry point holds its own copy for the life of the
// process; its address on the current device is looked up once per device
// and cached (the array's name in host code is not a device address).
static __device__ __align__(256) unsigned char scratch[HGA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

hga_status_t noalloc_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return HGA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return HGA_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HGA_OK;
}

static hga_status_t attend_bwd_impl(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                            const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                            const void* O, hga_strides_t os, const float* o_f32,
                            const void* dO, hga_strides_t dos,
                            const float* lse, int64_t q_begin, int64_t n_q, int64_t grad_begin,
                            const int32_t* sel_groups, const int32_t* n_sel_groups, float* dQ,
                            float* dK, float* dV, void* workspace, size_t workspace_bytes,
                            void* stream,
                                   const hga::AttnArgs* pre = nullptr, int64_t r_cap = 0) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_tensor(Q, qs, eb));
  HGA_TRY(check_tensor(K, ks, eb));
  HGA_TRY(check_tensor(V, vs, eb));
  HGA_TRY(check_tensor(O, os, eb));
  HGA_TRY(check_tensor(dO, dos, eb));
  HGA_TRY(check_rows(q_begin, n_q));
  if (grad_begin < 0 || grad_begin > q_begin || grad_begin % kChunk != 0) return HGA_ERR_INVALID_ARG;
  if (!lse || !n_sel_groups || (cfg->top_groups > 0 && !sel_groups)) return HGA_ERR_INVALID_ARG;
  if (!dQ || !dK || !dV || !aligned16(dQ) || !aligned16(dK) || !aligned16(dV))
    return HGA_ERR_INVALID_ARG;
  const size_t need = bwd_ws(cfg, q_begin, n_q, grad_begin);
  if (!workspace || workspace_bytes < need || !aligned16(workspace)) return HGA_ERR_WORKSPACE;
  AttnArgs a = attn_args(cfg, Q, qs, K, ks, V, vs, q_begin, n_q, sel_groups, n_sel_groups);
  if (o_f32 && !aligned16(o_f32)) return HGA_ERR_INVALID_ARG;
  a.O = O; a.o_tok = os.token; a.o_head = os.head;
  a.o32 = const_cast<float*>(o_f32);
  a.dO = dO; a.do_tok = dos.token; a.do_head = dos.head;
  a.lse = const_cast<float*>(lse);
  a.dQ = dQ; a.dK = dK; a.dV = dV;
  a.grad_begin = grad_begin;
  a.n_act_chunks = (int)((q_begin + n_q - grad_begin) / kChunk);
  a.dvec = static_cast<float*>(workspace);
  if (pre) {  // compact routed rows: dQ reads them, dK/dV reads the active-token view
    a.Kact = pre->Kact; a.ka_tok = pre->ka_tok; a.ka_head = pre->ka_head;
    a.Vact = pre->Vact; a.va_tok = pre->va_tok; a.va_head = pre->va_head;
    a.act_begin = pre->act_begin;
    a.r_cap = r_cap;
  }
  if (!a.Kact) {  // the dK/dV role reads its keys from K / V themselves
    a.Kact = K; a.ka_tok = ks.token; a.ka_head = ks.head;
    a.Vact = V; a.va_tok = vs.token; a.va_head = vs.head;
    a.act_begin = 0;
  }
  a.kv_parts = bwd_parts(cfg, q_begin);
  a.part_out = a.kv_parts > 1
      ? reinterpret_cast<float*>(static_cast<char*>(workspace) + bwd_dvec_bytes(cfg, n_q)) : nullptr;
  const hipError_t e = r_cap > 0 ? hga::launch_attend_gathered_bwd(a, cfg->dtype == HGA_BF16, cfg->head_dim,
                                                                   (hipStream_t)stream)
                                  : hga::launch_attend_bwd(a, cfg->dtype == HGA_BF16, cfg->head_dim,
                                                           (hipStream_t)stream);
  if (e != hipSuccess) return HGA_ERR_HIP;
  return HGA_OK;
}

}  // namespace

extern "C" {

const char* hga_status_string(hga_status_t s) {
  switch (s) {
    case HGA_OK: return "ok";
    case HGA_ERR_INVALID_ARG: return "invalid argument";
    case HGA_ERR_UNSUPPORTED: return "unsupported configuration";
    case HGA_ERR_WORKSPACE: return "workspace missing or too small";
    case HGA_ERR_HIP: return "HIP launch or runtime error";
  }
  return "unknown status";
}

size_t hga_workspace_size(const hga_config_t* cfg, int op, int64_t q_begin, int64_t n_q,
                          int64_t grad_begin) {
  if (check_cfg(cfg) != HGA_OK || check_rows(q_begin, n_q) != HGA_OK) return 0;
  if (op == HGA_OP_ROUTE) return route_ws(cfg, n_q);
  if (op == HGA_OP_BWD) {
    if (grad_begin < 0 || grad_begin > q_begin || grad_begin % kChunk != 0) return 0;
    return bwd_ws(cfg, q_begin, n_q, grad_begin);
  }
  return 0;
}

size_t hga_rows_workspace_size(const hga_config_t* cfg, int64_t n_q) {
  if (check_cfg(cfg) != HGA_OK || n_q <= 0 || n_q > hga::kRowsBwdMaxRows) return 0;
  return bwd_dvec_bytes(cfg, n_q);
}

hga_status_t hga_build_summaries(const hga_config_t* cfg, const void* K, hga_strides_t ks,
                                 int64_t t_begin, int64_t t_end, float* chunk_sum,
                                 int64_t chunk_cap, float* group_sum, int64_t group_cap,
                                 void* stream) {
  HGA_TRY(check_cfg(cfg));
  HGA_TRY(check_tensor(K, ks, elem_bytes(cfg)));
  if (t_begin < 0 || t_end <= t_begin || t_begin % kChunk != 0 || t_end > kMaxTokens) return HGA_ERR_INVALID_ARG;
  if (!chunk_sum || !group_sum || !aligned16(chunk_sum) || !aligned16(group_sum))
    return HGA_ERR_INVALID_ARG;
  if (chunk_cap < t_end / kChunk || group_cap < t_end / cfg->group_size) return HGA_ERR_INVALID_ARG;
  hga::SummaryArgs a = {};
  a.K = K; a.k_tok = ks.token; a.k_head = ks.head;
  a.t_begin = t_begin; a.t_end = t_end;
  a.chunk_sum = chunk_sum; a.chunk_cap = chunk_cap;
  a.group_sum = group_sum; a.group_cap = group_cap;
  a.n_kv_heads = cfg->n_kv_heads; a.head_dim = cfg->head_dim;
  a.group_shift = log2_exact(cfg->group_size);
  if (hga::launch_summaries(a, cfg->dtype == HGA_BF16, (hipStream_t)stream) != hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_route(const hga_config_t* cfg, const void* Q, hga_strides_t qs, int64_t q_begin,
                       int64_t n_q, const float* chunk_sum, int64_t chunk_cap,
                       const float* group_sum, int64_t group_cap, int32_t* sel_chunks,
                       int32_t* sel_groups, int32_t* n_sel_groups, void* workspace,
                       size_t workspace_bytes, void* stream) {
  hga::RouteArgs ra;
  int tb;
  HGA_TRY(route_args(cfg, Q, qs, q_begin, n_q, chunk_sum, chunk_cap, group_sum, group_cap, sel_chunks,
                     sel_groups, n_sel_groups, workspace, workspace_bytes, &ra, &tb));
  if (hga::launch_route(ra, cfg->dtype == HGA_BF16, cfg->head_dim, tb, (hipStream_t)stream) != hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_attend_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                            const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                            int64_t q_begin, int64_t n_q, const int32_t* sel_groups,
                            const int32_t* n_sel_groups, void* O, hga_strides_t os, float* lse,
                            float* o_f32, void* stream) {
  AttnArgs a;
  HGA_TRY(fwd_args(cfg, Q, qs, K, ks, V, vs, q_begin, n_q, sel_groups, n_sel_groups, O, os, lse, o_f32, &a));
  if (hga::launch_attend_fwd(a, cfg->dtype == HGA_BF16, cfg->head_dim, (hipStream_t)stream) !=
      hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_route_attend_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                  const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                  int64_t q_begin, int64_t n_q, const float* chunk_sum,
                                  int64_t chunk_cap, const float* group_sum, int64_t group_cap,
                                  int32_t* sel_chunks, int32_t* sel_groups, int32_t* n_sel_groups,
                                  void* O, hga_strides_t os, float* lse, float* o_f32,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  hga::RouteArgs ra;
  int tb;
  HGA_TRY(route_args(cfg, Q, qs, q_begin, n_q, chunk_sum, chunk_cap, group_sum, group_cap, sel_chunks,
                     sel_groups, n_sel_groups, workspace, workspace_bytes, &ra, &tb));
  AttnArgs a;
  HGA_TRY(fwd_args(cfg, Q, qs, K, ks, V, vs, q_begin, n_q, sel_groups, n_sel_groups, O, os, lse, o_f32, &a));
  const bool bf16 = cfg->dtype == HGA_BF16;
  const size_t route_lds = hga::route_lds_bytes(1, ra.score_stride, bf16);
  if (tb == 1 && hga::route_attend_fusable(a, route_lds)) {
    if (hga::launch_route_attend(ra, a, bf16, cfg->head_dim, route_lds, (hipStream_t)stream) != hipSuccess)
      return HGA_ERR_HIP;
    return HGA_OK;
  }
  if (hga::launch_route(ra, bf16, cfg->head_dim, tb, (hipStream_t)stream) != hipSuccess) return HGA_ERR_HIP;
  if (hga::launch_attend_fwd(a, bf16, cfg->head_dim, (hipStream_t)stream) != hipSuccess) return HGA_ERR_HIP;
  return HGA_OK;
}

// Rows per slot of the compact copies: every routed set fits.
int64_t min_r_cap(const hga_config_t* c) {
  const int64_t r = (int64_t)c->sink_tokens + c->local_tokens + (int64_t)c->top_groups * c->group_size;
  return (r + kChunk - 1) / kChunk * kChunk;
}

hga_status_t hga_gather_routed(const hga_config_t* cfg, const void* K, hga_strides_t ks,
                               const void* V, hga_strides_t vs, int64_t q_begin, int64_t n_q,
                               const int32_t* sel_groups, const int32_t* n_sel_groups,
                               void* Kc, void* Vc, int64_t r_cap, void* stream) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_tensor(K, ks, eb));
  HGA_TRY(check_tensor(V, vs, eb));
  HGA_TRY(check_rows(q_begin, n_q));
  if (!n_sel_groups || (cfg->top_groups > 0 && !sel_groups)) return HGA_ERR_INVALID_ARG;
  if (!Kc || !Vc || !aligned16(Kc) || !aligned16(Vc)) return HGA_ERR_INVALID_ARG;
  if (r_cap % kChunk != 0 || r_cap < min_r_cap(cfg)) return HGA_ERR_INVALID_ARG;
  AttnArgs a = attn_args(cfg, nullptr, hga_strides_t{1, 1}, K, ks, V, vs, q_begin, n_q, sel_groups,
                         n_sel_groups);
  a.r_cap = r_cap;
  if (hga::launch_gather(a, Kc, Vc, cfg->dtype == HGA_BF16, cfg->head_dim, (hipStream_t)stream) != hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_attend_gathered_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                     const void* Kc, const void* Vc, int64_t r_cap,
                                     int64_t q_begin, int64_t n_q, const int32_t* n_sel_groups,
                                     void* O, hga_strides_t os, float* lse, float* o_f32,
                                     void* stream) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_tensor(Q, qs, eb));
  HGA_TRY(check_tensor(O, os, eb));
  HGA_TRY(check_rows(q_begin, n_q));
  if (!lse || !n_sel_groups) return HGA_ERR_INVALID_ARG;
  if (!Kc || !Vc || !aligned16(Kc) || !aligned16(Vc)) return HGA_ERR_INVALID_ARG;
  if (r_cap % kChunk != 0 || r_cap < min_r_cap(cfg)) return HGA_ERR_INVALID_ARG;
  if (o_f32 && !aligned16(o_f32)) return HGA_ERR_INVALID_ARG;
  // the compact rows stand in for K and V; the strides are those of a
  // [rows][d] slot and are not used for addressing
  const hga_strides_t cs = {cfg->head_dim, cfg->head_dim};
  AttnArgs a = attn_args(cfg, Q, qs, Kc, cs, Vc, cs, q_begin, n_q, nullptr, n_sel_groups);
  a.r_cap = r_cap;
  a.Out = O; a.out_tok = os.token; a.out_head = os.head;
  a.lse = lse;
  a.o32 = o_f32;
  if (hga::launch_attend_gathered_fwd(a, cfg->dtype == HGA_BF16, cfg->head_dim, (hipStream_t)stream) !=
      hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_attend_bwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                            const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                            const void* O, hga_strides_t os, const float* o_f32,
                            const void* dO, hga_strides_t dos,
                            const float* lse, int64_t q_begin, int64_t n_q, int64_t grad_begin,
                            const int32_t* sel_groups, const int32_t* n_sel_groups, float* dQ,
                            float* dK, float* dV, void* workspace, size_t workspace_bytes,
                            void* stream) {
  return attend_bwd_impl(cfg, Q, qs, K, ks, V, vs, O, os, o_f32, dO, dos, lse, q_begin, n_q, grad_begin,
                         sel_groups, n_sel_groups, dQ, dK, dV, workspace, workspace_bytes, stream);
}

hga_status_t hga_attend_bwd_noalloc(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                    const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                    const void* O, hga_strides_t os, const float* o_f32,
                                    const void* dO, hga_strides_t dos,
                                    const float* lse, int64_t q_begin, int64_t n_q, int64_t grad_begin,
                                    const int32_t* sel_groups, const int32_t* n_sel_groups, float* dQ,
                                    float* dK, float* dV, void* stream) {
  // the size check comes first, so an oversized call returns before any HIP call
  HGA_TRY(check_cfg(cfg));
  HGA_TRY(check_rows(q_begin, n_q));
  if (grad_begin < 0 || grad_begin > q_begin || grad_begin % kChunk != 0) return HGA_ERR_INVALID_ARG;
  const size_t need = bwd_ws(cfg, q_begin, n_q, grad_begin);
  if (need > (size_t)HGA_NOALLOC_SCRATCH_BYTES) return HGA_ERR_WORKSPACE;
  void* ws = nullptr;
  HGA_TRY(noalloc_scratch(&ws));
  return attend_bwd_impl(cfg, Q, qs, K, ks, V, vs, O, os, o_f32, dO, dos, lse, q_begin, n_q, grad_begin,
                         sel_groups, n_sel_groups, dQ, dK, dV, ws, (size_t)HGA_NOALLOC_SCRATCH_BYTES, stream);
}

hga_status_t hga_route_rows(const hga_config_t* cfg, const void* Q, hga_strides_t qs, int64_t q_begin,
                            int64_t n_q, const float* chunk_sum, int64_t chunk_cap, const float* group_sum,
                            int64_t group_cap, int32_t* sel_chunks, int32_t* sel_groups,
                            int32_t* n_sel_groups, void* stream) {
  HGA_TRY(check_cfg(cfg));
  HGA_TRY(check_tensor(Q, qs, elem_bytes(cfg)));
  HGA_TRY(check_row_range(q_begin, n_q));
  const int64_t q_end = q_begin + n_q;
  if (!chunk_sum || !group_sum || !aligned16(chunk_sum) || !aligned16(group_sum))
    return HGA_ERR_INVALID_ARG;
  if (chunk_cap < q_end / kChunk || group_cap < q_end / cfg->group_size) return HGA_ERR_INVALID_ARG;
  if (!n_sel_groups || (cfg->top_chunks > 0 && !sel_chunks) || (cfg->top_groups > 0 && !sel_groups))
    return HGA_ERR_INVALID_ARG;
  const int gshift = log2_exact(cfg->group_size);
  const int gcand = cfg->top_chunks << (6 - gshift);
  if (gcand > kMaxGroupCand) return HGA_ERR_UNSUPPORTED;
  const int first_cand = (cfg->sink_tokens + kChunk - 1) / kChunk;
  // the last row's block has the longest candidate list
  const int64_t last_ls = ((q_end - 1) / kChunk + 1) * kChunk - cfg->local_tokens;
  const int n_cand_max = (int)(last_ls > 0 && last_ls / kChunk > first_cand ? last_ls / kChunk - first_cand : 0);
  hga::RouteArgs ra = {};
  ra.Q = Q; ra.q_tok = qs.token; ra.q_head = qs.head;
  ra.gqa = cfg->n_q_heads / cfg->n_kv_heads;
  ra.chunk_sum = chunk_sum; ra.chunk_cap = chunk_cap;
  ra.group_sum = group_sum; ra.group_cap = group_cap;
  ra.sel_chunks = sel_chunks; ra.sel_groups = sel_groups; ra.n_sel = n_sel_groups;
  ra.q_begin = q_begin; ra.n_qb = 0; ra.n_kv_heads = cfg->n_kv_heads;
  ra.top_chunks = cfg->top_chunks; ra.top_groups = cfg->top_groups; ra.group_shift = gshift;
  ra.sink_tokens = cfg->sink_tokens; ra.local_tokens = cfg->local_tokens;
  ra.first_cand = first_cand;
  if (hga::launch_route_rows(ra, n_q, n_cand_max, gcand, cfg->dtype == HGA_BF16, cfg->head_dim,
                             (hipStream_t)stream) != hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_attend_rows_fwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                 const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                 int64_t q_begin, int64_t n_q, const int32_t* sel_groups,
                                 const int32_t* n_sel_groups, void* O, hga_strides_t os, float* lse,
                                 float* o_f32, void* stream) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_tensor(Q, qs, eb));
  HGA_TRY(check_tensor(K, ks, eb));
  HGA_TRY(check_tensor(V, vs, eb));
  HGA_TRY(check_tensor(O, os, eb));
  HGA_TRY(check_row_range(q_begin, n_q));
  if (!lse || !n_sel_groups || (cfg->top_groups > 0 && !sel_groups)) return HGA_ERR_INVALID_ARG;
  AttnArgs a = attn_args(cfg, Q, qs, K, ks, V, vs, q_begin, n_q, sel_groups, n_sel_groups);
  if (o_f32 && !aligned16(o_f32)) return HGA_ERR_INVALID_ARG;
  a.n_qb = 0;
  a.Out = O; a.out_tok = os.token; a.out_head = os.head;
  a.lse = lse;
  a.o32 = o_f32;
  if (hga::launch_attend_rows_fwd(a, n_q, cfg->dtype == HGA_BF16, cfg->head_dim, (hipStream_t)stream) !=
      hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_attend_rows_bwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                 const void* K, hga_strides_t ks, const void* V, hga_strides_t vs,
                                 const void* O, hga_strides_t os, const float* o_f32,
                                 const void* dO, hga_strides_t dos, const float* lse, int64_t q_begin,
                                 int64_t n_q, int64_t grad_begin, const int32_t* sel_groups,
                                 const int32_t* n_sel_groups, float* dQ, float* dK, float* dV,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_tensor(Q, qs, eb));
  HGA_TRY(check_tensor(K, ks, eb));
  HGA_TRY(check_tensor(V, vs, eb));
  HGA_TRY(check_tensor(O, os, eb));
  HGA_TRY(check_tensor(dO, dos, eb));
  HGA_TRY(check_row_range(q_begin, n_q));
  if (grad_begin < 0 || grad_begin > q_begin || grad_begin % kChunk != 0) return HGA_ERR_INVALID_ARG;
  if (n_q > hga::kRowsBwdMaxRows) return HGA_ERR_UNSUPPORTED;
  if (!lse || !n_sel_groups || (cfg->top_groups > 0 && !sel_groups)) return HGA_ERR_INVALID_ARG;
  if (!dQ || !dK || !dV || !aligned16(dQ) || !aligned16(dK) || !aligned16(dV)) return HGA_ERR_INVALID_ARG;
  if (o_f32 && !aligned16(o_f32)) return HGA_ERR_INVALID_ARG;
  const size_t need = bwd_dvec_bytes(cfg, n_q);
  if (!workspace || workspace_bytes < need || !aligned16(workspace)) return HGA_ERR_WORKSPACE;
  AttnArgs a = attn_args(cfg, Q, qs, K, ks, V, vs, q_begin, n_q, sel_groups, n_sel_groups);
  a.n_qb = 0;
  a.O = O; a.o_tok = os.token; a.o_head = os.head;
  a.o32 = const_cast<float*>(o_f32);
  a.dO = dO; a.do_tok = dos.token; a.do_head = dos.head;
  a.lse = const_cast<float*>(lse);
  a.dQ = dQ; a.dK = dK; a.dV = dV;
  a.grad_begin = grad_begin;
  a.dvec = static_cast<float*>(workspace);
  if (hga::launch_attend_rows_bwd(a, n_q, cfg->dtype == HGA_BF16, cfg->head_dim, (hipStream_t)stream) !=
      hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

void* hga_host_device_view(const void* host_ptr) {
  if (!host_ptr) return nullptr;
  void* dev = nullptr;
  if (hipHostGetDevicePointer(&dev, const_cast<void*>(host_ptr), 0) != hipSuccess) {
    (void)hipGetLastError();  // leave no sticky error for the next call
    return nullptr;
  }
  return dev;
}

static hga_status_t cache_args(const hga_config_t* cfg, const hga_group_cache_t* cache, hga::CacheArgs* c) {
  if (!cache || !cache->slot_of || !cache->slot_chunk || !cache->cursor || !cache->groups ||
      !aligned16(cache->groups))
    return HGA_ERR_INVALID_ARG;
  if (cache->n_slots < 1 || cache->n_slots > hga::kMaxCacheSlots) return HGA_ERR_UNSUPPORTED;
  if (cache->chunk_cap < 1 || cache->chunk_cap > kMaxCacheChunks) return HGA_ERR_UNSUPPORTED;
  *c = hga::CacheArgs{};
  c->slot_of = cache->slot_of; c->slot_chunk = cache->slot_chunk; c->cursor = cache->cursor;
  c->groups = cache->groups; c->n_slots = cache->n_slots; c->chunk_cap = cache->chunk_cap;
  c->n_kv_heads = cfg->n_kv_heads; c->top_chunks = cfg->top_chunks;
  c->gpc_shift = 6 - log2_exact(cfg->group_size);
  return HGA_OK;
}

hga_status_t hga_group_cache_clear(const hga_config_t* cfg, const hga_group_cache_t* cache, void* stream) {
  HGA_TRY(check_cfg(cfg));
  hga::CacheArgs c;
  HGA_TRY(cache_args(cfg, cache, &c));
  if (hga::launch_cache_clear(c, (hipStream_t)stream) != hipSuccess) return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_route_cached(const hga_config_t* cfg, const void* Q, hga_strides_t qs, int64_t q_begin,
                              int64_t n_q, const float* chunk_sum, int64_t chunk_cap, const float* group_sum,
                              int64_t group_cap, const hga_group_cache_t* cache, int32_t* sel_chunks,
                              int32_t* sel_groups, int32_t* n_sel_groups, int32_t* cache_hit, void* workspace,
                              size_t workspace_bytes, void* stream) {
  hga::RouteArgs ra;
  int tb;
  HGA_TRY(route_args(cfg, Q, qs, q_begin, n_q, chunk_sum, chunk_cap, group_sum, group_cap, sel_chunks,
                     sel_groups, n_sel_groups, workspace, workspace_bytes, &ra, &tb));
  hga::CacheArgs c;
  HGA_TRY(cache_args(cfg, cache, &c));
  if (cache->chunk_cap < (q_begin + n_q) / kChunk) return HGA_ERR_INVALID_ARG;
  if (cfg->top_chunks > 0 && !cache_hit) return HGA_ERR_INVALID_ARG;
  ra.slot_of = cache->slot_of;
  ra.gcache = cache->groups;
  ra.gcache_cap = cache->n_slots << c.gpc_shift;
  ra.cache_hit = cfg->top_chunks > 0 ? cache_hit : nullptr;
  ra.chunk_cap = cache->chunk_cap;  // the slot map's row pitch (the chunk table's cap is not read past the chunks)
  if (chunk_cap != cache->chunk_cap) {
    // the routing reads chunk summaries with chunk_cap and the slot map with
    // the same field: they must agree
    return HGA_ERR_INVALID_ARG;
  }
  if (hga::launch_route(ra, cfg->dtype == HGA_BF16, cfg->head_dim, tb, (hipStream_t)stream) != hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_group_cache_update(const hga_config_t* cfg, const hga_group_cache_t* cache,
                                    const float* group_sum, int64_t group_cap, int64_t q_begin, int64_t n_q,
                                    const int32_t* sel_chunks, const int32_t* cache_hit, void* stream) {
  HGA_TRY(check_cfg(cfg));
  HGA_TRY(check_rows(q_begin, n_q));
  hga::CacheArgs c;
  HGA_TRY(cache_args(cfg, cache, &c));
  if (!group_sum || !aligned16(group_sum) || group_cap < (q_begin + n_q) / cfg->group_size)
    return HGA_ERR_INVALID_ARG;
  if (cache->chunk_cap < (q_begin + n_q) / kChunk) return HGA_ERR_INVALID_ARG;
  if (cfg->top_chunks == 0) return HGA_OK;  // nothing is ever chosen, nothing to bring in
  if (!sel_chunks || !cache_hit) return HGA_ERR_INVALID_ARG;
  c.group_sum = group_sum; c.group_cap = group_cap;
  c.sel_chunks = sel_chunks; c.cache_hit = cache_hit;
  c.n_qb = (int)(n_q / kChunk);
  if (hga::launch_cache_update(c, cfg->head_dim, (hipStream_t)stream) != hipSuccess) return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_gather_tiered(const hga_config_t* cfg, const void* K_hist, const void* V_hist,
                               hga_strides_t hs, int64_t hist_end, const void* K_act, const void* V_act,
                               hga_strides_t as, int64_t q_begin, int64_t n_q, const int32_t* sel_groups,
                               const int32_t* n_sel_groups, void* Kc, void* Vc, int64_t r_cap, void* stream) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_rows(q_begin, n_q));
  if (hist_end < 0 || hist_end > q_begin || hist_end % kChunk != 0) return HGA_ERR_INVALID_ARG;
  if (hist_end > 0) {
    HGA_TRY(check_tensor(K_hist, hs, eb));
    HGA_TRY(check_tensor(V_hist, hs, eb));
  }
  HGA_TRY(check_tensor(K_act, as, eb));
  HGA_TRY(check_tensor(V_act, as, eb));
  if (!n_sel_groups || (cfg->top_groups > 0 && !sel_groups)) return HGA_ERR_INVALID_ARG;
  if (!Kc || !Vc || !aligned16(Kc) || !aligned16(Vc)) return HGA_ERR_INVALID_ARG;
  if (r_cap % kChunk != 0 || r_cap < min_r_cap(cfg)) return HGA_ERR_INVALID_ARG;
  AttnArgs a = attn_args(cfg, nullptr, hga_strides_t{1, 1}, nullptr, hga_strides_t{1, 1}, nullptr,
                         hga_strides_t{1, 1}, q_begin, n_q, sel_groups, n_sel_groups);
  a.r_cap = r_cap;
  hga::TierArgs t = {};
  t.K_hist = hist_end > 0 ? K_hist : K_act; t.V_hist = hist_end > 0 ? V_hist : V_act;
  t.h_tok = hist_end > 0 ? hs.token : as.token; t.h_head = hist_end > 0 ? hs.head : as.head;
  t.K_act = K_act; t.V_act = V_act; t.a_tok = as.token; t.a_head = as.head;
  t.hist_end = hist_end;
  if (hga::launch_tier_gather(a, t, Kc, Vc, cfg->dtype == HGA_BF16, cfg->head_dim, (hipStream_t)stream) !=
      hipSuccess)
    return HGA_ERR_HIP;
  return HGA_OK;
}

hga_status_t hga_attend_gathered_bwd(const hga_config_t* cfg, const void* Q, hga_strides_t qs,
                                     const void* Kc, const void* Vc, int64_t r_cap, const void* K_act,
                                     const void* V_act, hga_strides_t as, int64_t act_begin,
                                     const void* O, hga_strides_t os, const float* o_f32,
                                     const void* dO, hga_strides_t dos, const float* lse, int64_t q_begin,
                                     int64_t n_q, int64_t grad_begin, const int32_t* sel_groups,
                                     const int32_t* n_sel_groups, float* dQ, float* dK, float* dV,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  HGA_TRY(check_cfg(cfg));
  const int eb = elem_bytes(cfg);
  HGA_TRY(check_rows(q_begin, n_q));
  if (!Kc || !Vc || !aligned16(Kc) || !aligned16(Vc)) return HGA_ERR_INVALID_ARG;
  if (r_cap % kChunk != 0 || r_cap < min_r_cap(cfg)) return HGA_ERR_INVALID_ARG;
  HGA_TRY(check_tensor(K_act, as, eb));
  HGA_TRY(check_tensor(V_act, as, eb));
  if (act_begin < 0 || act_begin % kChunk != 0 || act_begin > q_begin) return HGA_ERR_INVALID_ARG;
  if (grad_begin < act_begin) return HGA_ERR_INVALID_ARG;  // dK/dV rows must be device rows
  hga::AttnArgs pre = {};
  pre.Kact = K_act; pre.ka_tok = as.token; pre.ka_head = as.head;
  pre.Vact = V_act; pre.va_tok = as.token; pre.va_head = as.head;
  pre.act_begin = act_begin;
  // compact rows stand in for K and V (strides of a [rows][d] slot; not used
  // for addressing)
  const hga_strides_t cs = {cfg->head_dim, cfg->head_dim};
  return attend_bwd_impl(cfg, Q, qs, Kc, cs, Vc, cs, O, os, o_f32, dO, dos, lse, q_begin, n_q, grad_begin,
                         sel_groups, n_sel_groups, dQ, dK, dV, workspace, workspace_bytes, stream, &pre, r_cap);
}

}  // extern "C"
