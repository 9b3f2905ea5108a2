// Per-query routing and attention: every query row routes on its own (the
// block descriptor of Sec. 2.1 item 1 taken over a block of one query), and
// attends its own routed set. This is routing at generation time, one or a
// few queries per call (Sec. 1, last result: routed generation; Sec. 7),
// and, applied to every row of a training segment, a strictly causal
// variant of the method (Sec. 6.1: with a routing decision shared by a whole
// block, an early query's attended set depends on later queries; here it
// depends only on its own row and on keys before its block).
//
// A query keeps the windows and the candidate chunks of the 64-token block
// holding it (sink window, local window ending at the block end, chunks
// closed before the local window) and attends only tokens up to its own
// position, so rows after it are never read.
//
// Routing: one workgroup of four waves per (four consecutive query rows, or
// one row when the call is too small to fill the chip that way, kv head). A row's descriptor is the exact
// float64 mean of its G query-head rows; chunk and group scores (one
// candidate per thread, against every row of the workgroup) are float64 FMA
// chains over the float32 summaries, ranked by wave_top_k, one wave per row
// (larger score first, lower index on ties; sets returned ascending).
//
// Attention: one workgroup of four waves per (query row, kv head), all G
// query heads together. A single query row is no dense contraction, so the
// work stays on the vector units: lane = key for the scores (each lane reads
// its key's K and V rows), an online softmax with wave-uniform maxima, and
// lane = head-dim slice for P.V over the tile's V rows staged in LDS. The
// four waves take every fourth 64-key tile of the routed set and merge their
// partial softmax states at the end.
#include "route_device.h"

namespace hga {

// ---------------------------------------------------------------- routing

template <typename T, int D>
__device__ inline float load_elem(const char* p) {
  if constexpr (Elem<T>::kBytes == 2) return bf16_bits_to_float(*reinterpret_cast<const uint16_t*>(p));
  else return *reinterpret_cast<const float*>(p);
}

// Float64 dot product of the descriptor with summary row r of a quad-major
// table (two FMA chains over the even and odd head-dim elements).
template <int D>
__device__ inline double summary_dot(const float* table, int64_t r, int64_t cap, const double* q) {
  const f32x4* t = reinterpret_cast<const f32x4*>(table) + r;
  f32x4 v[D / 4];
#pragma unroll
  for (int k = 0; k < D / 4; ++k) v[k] = t[(int64_t)k * cap];  // every load in flight
  double a0 = 0.0, a1 = 0.0;
#pragma unroll
  for (int k = 0; k < D / 4; ++k) {
    a0 = fma((double)v[k][0], q[4 * k], a0);
    a1 = fma((double)v[k][1], q[4 * k + 1], a1);
    a0 = fma((double)v[k][2], q[4 * k + 2], a0);
    a1 = fma((double)v[k][3], q[4 * k + 3], a1);
    // keep each quad's conversions and descriptor reads with it (hoisting
    // them all ahead doubles the live registers)
    __builtin_amdgcn_sched_barrier(0);
  }
  return a0 + a1;
}

// Float64 dots of summary row r with the descriptors q[0..nv): per
// descriptor the two FMA chains of summary_dot, in the same order, with the
// row read and converted once for all of them.
template <int D, int RB>
__device__ inline void summary_dots(const float* table, int64_t r, int64_t cap, const double (*q)[D], int nv,
                                    double (&out)[RB]) {
  const f32x4* t = reinterpret_cast<const f32x4*>(table) + r;
  f32x4 v[D / 4];
#pragma unroll
  for (int k = 0; k < D / 4; ++k) v[k] = t[(int64_t)k * cap];  // every load in flight
  double a0[RB], a1[RB];
#pragma unroll
  for (int w = 0; w < RB; ++w) a0[w] = a1[w] = 0.0;
#pragma unroll
  for (int k = 0; k < D / 4; ++k) {
    const double x0 = v[k][0], x1 = v[k][1], x2 = v[k][2], x3 = v[k][3];
#pragma unroll
    for (int w = 0; w < RB; ++w) {
      if (w < nv) {
        a0[w] = fma(x0, q[w][4 * k], a0[w]);
        a1[w] = fma(x1, q[w][4 * k + 1], a1[w]);
        a0[w] = fma(x2, q[w][4 * k + 2], a0[w]);
        a1[w] = fma(x3, q[w][4 * k + 3], a1[w]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int w = 0; w < RB; ++w) out[w] = a0[w] + a1[w];
}

// One workgroup of four waves per (RB consecutive query rows, kv head).
// Every chunk-summary row the call scores is read once per workgroup and
// scored against the RB row descriptors (rows of one block share their
// candidate list; rows of two blocks score the longer list, each keeping its
// own prefix); wave w then selects for row w. Candidates are taken in rounds
// of RR: after each round a row's selection is the top-k_c of [its running
// selection | the round's scores]. The kept entries sit ahead of the round's
// and have lower chunk ids, so positions keep chunk order, ties still go to
// the lower chunk, and the selection is the whole list's. `stride`: doubles
// of dynamic LDS per row.
template <int RB>
struct RowsRoute {
  static constexpr int RR = RB == 1 ? kRowsRouteRound : 512;
};

template <typename T, int D, int RB>
__global__ __launch_bounds__(256) void route_rows_kernel(RouteArgs a, int64_t n_rows, int stride) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int RR = RowsRoute<RB>::RR;
  static_assert(RB <= 4, "one selecting wave per row");
  extern __shared__ double dyn[];  // per row: [kept | the round's scores], then its group scores
  __shared__ __attribute__((aligned(16))) double s_q[RB][D];
  __shared__ TopKScratch s_tk[RB];
  __shared__ double s_kv[RB][64];
  __shared__ int s_ki[RB][64];
  __shared__ int s_chunks[RB][64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t row0 = (int64_t)(blockIdx.x / a.n_kv_heads) * RB;
  const int nv = (int)(n_rows - row0 < RB ? n_rows - row0 : RB);  // rows of this workgroup
  const int G = a.gqa;

  // descriptors: the mean of each row's G head rows of kv head h (a sum of G
  // bf16 or float32 values and a division by a power of two: exact)
  for (int x = tid; x < RB * D; x += 256) {
    const int w = x / D, e = x % D;
    double s = 0.0;
    if (w < nv) {
      const char* qrow = static_cast<const char*>(a.Q) + ((row0 + w) * a.q_tok + (int64_t)h * G * a.q_head) * EB;
      for (int g = 0; g < G; ++g) s += (double)load_elem<T, D>(qrow + ((int64_t)g * a.q_head + e) * EB);
      s /= (double)G;
    }
    s_q[w][e] = s;
  }
  __syncthreads();

  // candidates [c_lo, c_lo + n) of row w: a prefix of the longest list
  const int c_lo = a.first_cand;
  auto n_cand_of = [&](int w) {
    return max(0, last_cand((a.q_begin + row0 + w) / 64, a.local_tokens) - c_lo);
  };
  int n_max = 0;
  for (int w = 0; w < nv; ++w) n_max = max(n_max, n_cand_of(w));
  const int my_n = wave < nv ? n_cand_of(wave) : 0;
  const float* cs = a.chunk_sum + quad_off(h, 0, 0, D, a.chunk_cap);
  const int n_rounds = max(1, (n_max + RR - 1) / RR);
  double* mine = dyn + wave * stride;  // this wave's row (wave < nv)
  int n_kept = 0;
  for (int r = 0; r < n_rounds; ++r) {
    const int nr = max(0, min(RR, n_max - r * RR));
    const int r0 = c_lo + r * RR;
    for (int i0 = 0; i0 < nr; i0 += 256) {
      const int i = i0 + tid;
      double v[RB];
      summary_dots<D, RB>(cs, r0 + min(i, nr - 1), a.chunk_cap, s_q, nv, v);
      if (i < nr) {
#pragma unroll
        for (int w = 0; w < RB; ++w)
          if (w < nv) dyn[w * stride + 64 + i] = no_nan(v[w]);
      }
    }
    __syncthreads();
    const int nr_w = max(0, min(RR, my_n - r * RR));
    if (wave < nv && nr_w > 0) {
      double* base = mine + 64 - n_kept;
      if (lane < n_kept) base[lane] = s_kv[wave][lane];
      __builtin_amdgcn_wave_barrier();
      const int n = n_kept + nr_w;
      const int pc = wave_top_k(base, n, a.top_chunks, lane, s_tk[wave]);
      const int k_eff = min(a.top_chunks, n);
      double v = 0.0;
      int idx = -1;
      if (lane < k_eff) {  // pc is a position only on those lanes
        v = base[pc];
        idx = pc < n_kept ? s_ki[wave][pc] : r0 + (pc - n_kept);
      }
      __builtin_amdgcn_wave_barrier();
      if (lane < k_eff) {
        s_kv[wave][lane] = v;
        s_ki[wave][lane] = idx;
      }
      n_kept = k_eff;
    }
    __syncthreads();  // the round's scores are read: the next round may overwrite them
  }
  const int kc_eff = min(a.top_chunks, my_n);  // this wave's row
  const int64_t slot = (row0 + wave) * a.n_kv_heads + h;
  if (wave < nv) {
    const int chunk = lane < kc_eff ? s_ki[wave][lane] : -1;
    if (lane < a.top_chunks) a.sel_chunks[slot * a.top_chunks + lane] = chunk;
    s_chunks[wave][lane] = lane < kc_eff ? chunk : 0;
  }
  __syncthreads();

  // group scores over every group of each row's chosen chunks (ascending
  // ids): item f of row w is group f of its list
  const int gpc_shift = 6 - a.group_shift;
  const int gmask = (1 << gpc_shift) - 1;
  const int gslot = a.top_chunks << gpc_shift;  // items per row
  if (a.top_groups > 0 && gslot > 0) {
    const float* gs = a.group_sum + quad_off(h, 0, 0, D, a.group_cap);
    for (int f0 = 0; f0 < nv * gslot; f0 += 256) {
      const int fa = f0 + tid, w = fa / gslot, f = fa - w * gslot;
      if (w < nv && f < (min(a.top_chunks, n_cand_of(w)) << gpc_shift)) {
        const int64_t j = ((int64_t)s_chunks[w][f >> gpc_shift] << gpc_shift) + (f & gmask);
        dyn[w * stride + f] = no_nan(summary_dot<D>(gs, j, a.group_cap, s_q[w]));
      }
    }
  }
  __syncthreads();
  if (wave >= nv) return;
  const int n_gc = kc_eff << gpc_shift;
  if (a.top_groups > 0) {
    const int kg_eff = min(a.top_groups, n_gc);
    const int pg = wave_top_k(mine, n_gc, a.top_groups, lane, s_tk[wave]);
    const int pgs = lane < kg_eff ? pg : 0;  // pg is a position only on those lanes
    const int gid = (s_chunks[wave][pgs >> gpc_shift] << gpc_shift) + (pgs & gmask);
    if (lane < a.top_groups) a.sel_groups[slot * a.top_groups + lane] = lane < kg_eff ? gid : -1;
    if (lane == 0) a.n_sel[slot] = kg_eff;
  } else if (lane == 0) {
    a.n_sel[slot] = 0;
  }
}

// Rows per routing workgroup: four when the call still fills the chip with
// (four rows, kv head) workgroups (each summary row read then serves four
// rows), else one (decode steps and short calls keep one workgroup per row).
static int route_rows_per_wg(int64_t n_rows, int n_kv_heads) {
  return (n_rows + 3) / 4 * n_kv_heads >= 256 ? 4 : 1;
}

hipError_t launch_route_rows(const RouteArgs& a, int64_t n_rows, int n_cand_max, int group_cand, bool bf16,
                             int head_dim, hipStream_t s) {
  const int rb = route_rows_per_wg(n_rows, a.n_kv_heads);
  const int rr = rb == 1 ? RowsRoute<1>::RR : RowsRoute<4>::RR;
  const int nc = 64 + (n_cand_max < rr ? n_cand_max : rr);
  const int stride = nc > group_cand ? nc : group_cand;
  const size_t lds = (size_t)rb * stride * sizeof(double);
  const dim3 grid((unsigned)((n_rows + rb - 1) / rb * a.n_kv_heads)), block(256);
#define HGA_RR(T, D, RB) hipLaunchKernelGGL((route_rows_kernel<T, D, RB>), grid, block, lds, s, a, n_rows, stride)
  if (rb == 1) {
    if (!bf16) HGA_RR(float, 64, 1);
    else if (head_dim == 64) HGA_RR(__bf16, 64, 1);
    else HGA_RR(__bf16, 128, 1);
  } else {
    if (!bf16) HGA_RR(float, 64, 4);
    else if (head_dim == 64) HGA_RR(__bf16, 64, 4);
    else HGA_RR(__bf16, 128, 4);
  }
#undef HGA_RR
  return hipGetLastError();
}

// ---------------------------------------------------------------- attention

// Wave-wide maximum and sum, the same value in every lane: DPP steps inside
// each 16-lane row (swap neighbours, swap pairs, mirror each half-row,
// mirror the row), then the four rows' values read as scalars. No step goes
// through the LDS crossbar.
template <int CTRL>
__device__ inline float dpp_src(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
__device__ inline float row_lane(float x, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), l));
}
__device__ inline float wave_max(float v) {
  v = fmaxf(v, dpp_src<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_src<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_src<0x141>(v));  // row_half_mirror
  v = fmaxf(v, dpp_src<0x140>(v));  // row_mirror
  return fmaxf(fmaxf(row_lane(v, 0), row_lane(v, 16)), fmaxf(row_lane(v, 32), row_lane(v, 48)));
}
__device__ inline float wave_sum(float v) {
  v += dpp_src<0xB1>(v);
  v += dpp_src<0x4E>(v);
  v += dpp_src<0x141>(v);
  v += dpp_src<0x140>(v);
  return (row_lane(v, 0) + row_lane(v, 16)) + (row_lane(v, 32) + row_lane(v, 48));
}

// Token at position p of a row's routed set [sink | selected groups | local
// window up to the row].
__device__ inline int64_t row_token(int p, int n_sink, int n_grp_tok, int64_t ls, const int32_t* sel,
                                    int gshift) {
  if (p < n_sink) return p;
  if (p < n_sink + n_grp_tok) {
    const int q = p - n_sink;
    return ((int64_t)sel[q >> gshift] << gshift) + (q & ((1 << gshift) - 1));
  }
  return ls + (p - n_sink - n_grp_tok);
}

// The routed set of query row `row` for kv head h.
struct RowSet {
  int64_t pos, ls;
  int n_sink, n_grp_tok, R;
  const int32_t* sel;
};

__device__ inline RowSet row_set(const AttnArgs& a, int64_t row, int h) {
  RowSet r;
  r.pos = a.q_begin + row;
  const int64_t block_end = (r.pos / 64 + 1) * 64;
  r.ls = block_end - a.local_tokens > 0 ? block_end - a.local_tokens : 0;
  r.n_sink = (int)min((int64_t)a.sink_tokens, r.ls);
  const int64_t slot = row * a.n_kv_heads + h;
  const int n_sel = a.top_groups > 0 ? a.n_sel[slot] : 0;
  r.n_grp_tok = n_sel << a.group_shift;
  r.R = r.n_sink + r.n_grp_tok + (int)(r.pos + 1 - r.ls);
  r.sel = a.top_groups > 0 ? a.sel_groups + slot * a.top_groups : nullptr;
  return r;
}

template <typename T, int D, int G>
__global__ __launch_bounds__(256) void attend_rows_fwd_kernel(AttnArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E = D / 64;             // head-dim elements of a lane in P.V
  constexpr int NP = D * EB / 16;       // 16-byte pieces of a key row
  constexpr int EP = 16 / EB;           // elements per piece
  constexpr int VP = D * EB + 16;       // LDS pitch of a staged V row (padded against bank conflicts)
  __shared__ __attribute__((aligned(16))) float s_q[G][D];
  __shared__ float s_m[4][G], s_l[4][G];
  __shared__ float s_o[4][G][D];
  __shared__ __attribute__((aligned(16))) char s_v[4][64 * VP];  // each wave's current V tile, row = key
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t row = blockIdx.x / a.n_kv_heads;
  const char* Qb = static_cast<const char*>(a.Q);
  const char* Kb = static_cast<const char*>(a.K);
  const char* Vb = static_cast<const char*>(a.V);

  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, e = x % D;
    s_q[g][e] = load_elem<T, D>(Qb + (row * a.q_tok + (int64_t)(h * G + g) * a.q_head + e) * EB);
  }
  const RowSet rs = row_set(a, row, h);
  __syncthreads();

  float m[G], l[G], o[G][E];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -__builtin_inff();
    l[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) o[g][e] = 0.0f;
  }
  const int64_t k_stride = a.k_tok * EB, v_stride = a.v_tok * EB;
  const int64_t k_head = (int64_t)h * a.k_head * EB, v_head = (int64_t)h * a.v_head * EB;
  for (int tb = wave * 64; tb < rs.R; tb += 256) {
    const int p = tb + lane;
    const bool valid = p < rs.R;
    const int64_t t = row_token(min(p, rs.R - 1), rs.n_sink, rs.n_grp_tok, rs.ls, rs.sel, a.group_shift);
    // scores of this lane's key for the G query heads; its V row goes out
    // with its K row and is staged in LDS for P.V
    const char* kr = row_ptr(Kb, t, k_stride) + k_head;
    const char* vrow = row_ptr(Vb, t, v_stride) + v_head;
    u32x4 kw[NP], vw[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) kw[c] = *reinterpret_cast<const u32x4*>(kr + 16 * c);
#pragma unroll
    for (int c = 0; c < NP; ++c) vw[c] = *reinterpret_cast<const u32x4*>(vrow + 16 * c);
    float s[G];
#pragma unroll
    for (int g = 0; g < G; ++g) s[g] = 0.0f;
#pragma unroll
    for (int c = 0; c < NP; ++c) {
      float kx[EP];
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        if constexpr (EB == 2) kx[e] = bf16_bits_to_float((kw[c][e >> 1] >> ((e & 1) * 16)) & 0xffffu);
        else kx[e] = __uint_as_float(kw[c][e]);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
#pragma unroll
        for (int e4 = 0; e4 < EP / 4; ++e4) {
          const f32x4 qq = *reinterpret_cast<const f32x4*>(&s_q[g][c * EP + 4 * e4]);
#pragma unroll
          for (int e = 0; e < 4; ++e) s[g] = fmaf(qq[e], kx[4 * e4 + e], s[g]);
        }
      }
      // one piece at a time: its conversions and query reads stay with it
      __builtin_amdgcn_sched_barrier(0);
    }
    // online softmax in log2 units; the maximum is uniform over the wave
    float pr[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sg = valid ? s[g] * a.scale_log2 : -__builtin_inff();
      const float mn = fmaxf(m[g], wave_max(sg));
      const float alpha = exp2f(m[g] - mn);
      pr[g] = exp2f(sg - mn);
      l[g] = l[g] * alpha + pr[g];
#pragma unroll
      for (int e = 0; e < E; ++e) o[g][e] *= alpha;
      m[g] = mn;
    }
    // P.V: the tile's V rows through LDS (row = key), then lane = head-dim
    // slice reads each key's slice (consecutive lanes, consecutive words)
    char* sv = s_v[wave];
#pragma unroll
    for (int c = 0; c < NP; ++c) *reinterpret_cast<u32x4*>(sv + lane * VP + 16 * c) = vw[c];
    __builtin_amdgcn_wave_barrier();
    const int nk = min(64, rs.R - tb);
#pragma unroll 1
    for (int j0 = 0; j0 < nk; j0 += 8) {
      float vv[8][E];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) vv[u][e] = load_elem<T, D>(sv + (j0 + u) * VP + (lane * E + e) * EB);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (j0 + u < nk) {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float pj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pr[g]), j0 + u));
#pragma unroll
            for (int e = 0; e < E; ++e) o[g][e] = fmaf(pj, vv[u][e], o[g][e]);
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  // merge the four waves' partial softmax states
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float lt = wave_sum(l[g]);
    if (lane == 0) {
      s_m[wave][g] = m[g];
      s_l[wave][g] = lt;
    }
#pragma unroll
    for (int e = 0; e < E; ++e) s_o[wave][g][lane * E + e] = o[g][e];
  }
  __syncthreads();
  char* Ob = static_cast<char*>(a.Out);
  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, e = x % D;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][g]);
    float num = 0.0f, den = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = s_m[w][g] == -__builtin_inff() ? 0.0f : exp2f(s_m[w][g] - M);
      num = fmaf(f, s_o[w][g][e], num);
      den = fmaf(f, s_l[w][g], den);
    }
    const float out = num / den;
    char* op = Ob + (row * a.out_tok + (int64_t)(h * G + g) * a.out_head + e) * EB;
    if constexpr (EB == 2) *reinterpret_cast<uint16_t*>(op) = (uint16_t)float_to_bf16_bits(out);
    else *reinterpret_cast<float*>(op) = out;
    if (a.o32) a.o32[(row * a.n_q_heads + h * G + g) * D + e] = out;
    if (e == 0) a.lse[row * a.n_q_heads + h * G + g] = (M + log2f(den)) * kLn2;
  }
}

// bf16: the scores and P.V on the matrix cores, with the 4x4x4 product that
// computes sixteen independent 4 x 4 blocks per instruction
// (v_mfma_f32_4x4x4_16b_bf16): lanes 4b .. 4b+3 hold block b; lane 4b+i gives
// row i of A and lane 4b+j column j of B (four k values each), and lane 4b+j
// receives column j of the block's 4 x 4 result.
//  - S: the query heads are the rows of A (four per product, zero rows past
//    G), the keys the columns of B (lane = key, its own K row) and the head
//    dim the k axis: lane = key receives its key's score for four heads, the
//    layout the softmax below works in.
//  - P.V: the heads are again the rows (P from LDS, rounded to bf16 as in
//    the block kernels' P.V), the tile's keys the k axis, and the head dim
//    the columns: sixteen blocks of four columns per product, B read from the
//    row-major V tile with the LDS transpose load. Lane l receives column
//    64 dh + l of O for four heads.
template <int D, int G>
__global__ __launch_bounds__(256) void attend_rows_fwd_mfma_kernel(AttnArgs a) {
  constexpr int NG = (G + 3) / 4;  // four-head row groups of A
  constexpr int GR = 4 * NG;       // rows of A (heads past G are zero)
  constexpr int NP = D * 2 / 16;   // 16-byte pieces of a key row
  constexpr int NKS = D / 4;       // k steps of S
  constexpr int NDH = D / 64;      // 64-column slices of O
  constexpr int VP = D * 2 + 16;   // LDS pitch of a staged V row (padded against bank conflicts)
  __shared__ __attribute__((aligned(16))) uint16_t s_q[GR][D];      // bf16 query rows of the G heads
  __shared__ __attribute__((aligned(16))) uint16_t s_p[4][GR][64];  // each wave's P, bf16, [head][key]
  __shared__ float s_m[4][G], s_l[4][G];
  // each wave's current half tile of V rows (32 keys), row = key; after the
  // tiles, its partial O (about 38 KB of LDS in all: three workgroups per CU)
  __shared__ __attribute__((aligned(16))) char s_v[4][32 * VP];
  static_assert(G * D * 4 <= 32 * VP, "a wave's partial O fits its V buffer");
  typedef __attribute__((address_space(3))) s16x4* lds_s4;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t row = blockIdx.x / a.n_kv_heads;
  const char* Qb = static_cast<const char*>(a.Q);
  const char* Kb = static_cast<const char*>(a.K);
  const char* Vb = static_cast<const char*>(a.V);

  for (int x = tid; x < GR * D; x += 256) {
    const int g = x / D, e = x % D;
    s_q[g][e] = g < G ? *reinterpret_cast<const uint16_t*>(Qb + (row * a.q_tok + (int64_t)(h * G + g) * a.q_head + e) * 2)
                      : (uint16_t)0;
  }
  if constexpr (GR > G) {
    for (int x = tid; x < 4 * (GR - G) * 64; x += 256) s_p[x / ((GR - G) * 64)][G + (x / 64) % (GR - G)][x % 64] = 0;
  }
  const RowSet rs = row_set(a, row, h);
  __syncthreads();

  float m[G], l[G];
  f32x4 oacc[NG][NDH];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -__builtin_inff();
    l[g] = 0.0f;
  }
#pragma unroll
  for (int ng = 0; ng < NG; ++ng)
#pragma unroll
    for (int dh = 0; dh < NDH; ++dh) oacc[ng][dh] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  const int64_t k_stride = a.k_tok * 2, v_stride = a.v_tok * 2;
  const int64_t k_head = (int64_t)h * a.k_head * 2, v_head = (int64_t)h * a.v_head * 2;
  char* sv = s_v[wave];
  uint16_t(*sp)[64] = s_p[wave];
  for (int tb = wave * 64; tb < rs.R; tb += 256) {
    const int p = tb + lane;
    const bool valid = p < rs.R;
    const int64_t t = row_token(min(p, rs.R - 1), rs.n_sink, rs.n_grp_tok, rs.ls, rs.sel, a.group_shift);
    const char* kr = row_ptr(Kb, t, k_stride) + k_head;
    const char* vrow = row_ptr(Vb, t, v_stride) + v_head;
    u32x4 kw[NP], vw[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) kw[c] = *reinterpret_cast<const u32x4*>(kr + 16 * c);
#pragma unroll
    for (int c = 0; c < NP; ++c) vw[c] = *reinterpret_cast<const u32x4*>(vrow + 16 * c);
    // S: this lane's key against the G heads, four heads per product
    f32x4 sacc[NG];
#pragma unroll
    for (int ng = 0; ng < NG; ++ng) sacc[ng] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const u32x4 pc = kw[ks / 2];
      const s16x4 kb = __builtin_bit_cast(s16x4, uint2{pc[2 * (ks % 2)], pc[2 * (ks % 2) + 1]});
#pragma unroll
      for (int ng = 0; ng < NG; ++ng) {
        const s16x4 qa = *reinterpret_cast<const s16x4*>(&s_q[4 * ng + (lane & 3)][4 * ks]);
        sacc[ng] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(qa, kb, sacc[ng], 0, 0, 0);
      }
    }
    // online softmax in log2 units; the maximum is uniform over the wave
    float pr[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sg = valid ? sacc[g / 4][g % 4] * a.scale_log2 : -__builtin_inff();
      const float mn = fmaxf(m[g], wave_max(sg));
      const float alpha = exp2f(m[g] - mn);
      pr[g] = exp2f(sg - mn);
      l[g] = l[g] * alpha + pr[g];
#pragma unroll
      for (int dh = 0; dh < NDH; ++dh) oacc[g / 4][dh][g % 4] *= alpha;
      m[g] = mn;
    }
    // P (bf16) and the tile's V rows through LDS
#pragma unroll
    for (int g = 0; g < G; ++g) sp[g][lane] = (uint16_t)float_to_bf16_bits(pr[g]);
    // P.V over the tile's 64 keys in two halves of 32, each half's V rows
    // staged by its own lanes, four keys per k step
    const int i = lane & 15, col0 = 16 * (lane >> 4) + 4 * (i & 3);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      if ((lane >> 5) == hf) {
#pragma unroll
        for (int c = 0; c < NP; ++c) *reinterpret_cast<u32x4*>(sv + (lane & 31) * VP + 16 * c) = vw[c];
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll 4
      for (int k8 = 0; k8 < 8; ++k8) {
        const int kk = 8 * hf + k8;
        s16x4 pa[NG];
#pragma unroll
        for (int ng = 0; ng < NG; ++ng) pa[ng] = *reinterpret_cast<const s16x4*>(&sp[4 * ng + (lane & 3)][4 * kk]);
#pragma unroll
        for (int dh = 0; dh < NDH; ++dh) {
          const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_s4)(sv + (4 * k8 + (i >> 2)) * VP + (64 * dh + col0) * 2));
#pragma unroll
          for (int ng = 0; ng < NG; ++ng) oacc[ng][dh] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(pa[ng], vb, oacc[ng][dh], 0, 0, 0);
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  // merge the four waves' partial softmax states; a wave's O goes to its own
  // V buffer, which only it has used
  float* so = reinterpret_cast<float*>(sv);
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float lt = wave_sum(l[g]);
    if (lane == 0) {
      s_m[wave][g] = m[g];
      s_l[wave][g] = lt;
    }
#pragma unroll
    for (int dh = 0; dh < NDH; ++dh) so[g * D + 64 * dh + lane] = oacc[g / 4][dh][g % 4];
  }
  __syncthreads();
  char* Ob = static_cast<char*>(a.Out);
  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, e = x % D;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][g]);
    float num = 0.0f, den = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = s_m[w][g] == -__builtin_inff() ? 0.0f : exp2f(s_m[w][g] - M);
      num = fmaf(f, reinterpret_cast<const float*>(s_v[w])[g * D + e], num);
      den = fmaf(f, s_l[w][g], den);
    }
    const float out = num / den;
    char* op = Ob + (row * a.out_tok + (int64_t)(h * G + g) * a.out_head + e) * 2;
    *reinterpret_cast<uint16_t*>(op) = (uint16_t)float_to_bf16_bits(out);
    if (a.o32) a.o32[(row * a.n_q_heads + h * G + g) * D + e] = out;
    if (e == 0) a.lse[row * a.n_q_heads + h * G + g] = (M + log2f(den)) * kLn2;
  }
}

template <typename T, int D>
hipError_t rows_fwd_g(const AttnArgs& a, int64_t n_rows, hipStream_t s) {
  const dim3 grid((unsigned)(n_rows * a.n_kv_heads)), block(256);
  if constexpr (Elem<T>::kBytes == 2) {
    switch (a.gqa) {
      case 1: hipLaunchKernelGGL((attend_rows_fwd_mfma_kernel<D, 1>), grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL((attend_rows_fwd_mfma_kernel<D, 2>), grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL((attend_rows_fwd_mfma_kernel<D, 4>), grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL((attend_rows_fwd_mfma_kernel<D, 8>), grid, block, 0, s, a); break;
    }
  } else {
    switch (a.gqa) {
      case 1: hipLaunchKernelGGL((attend_rows_fwd_kernel<T, D, 1>), grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL((attend_rows_fwd_kernel<T, D, 2>), grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL((attend_rows_fwd_kernel<T, D, 4>), grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL((attend_rows_fwd_kernel<T, D, 8>), grid, block, 0, s, a); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_attend_rows_fwd(const AttnArgs& a, int64_t n_rows, bool bf16, int head_dim, hipStream_t s) {
  if (!bf16) return rows_fwd_g<float, 64>(a, n_rows, s);  // float32 is built for head_dim 64 only
  return head_dim == 64 ? rows_fwd_g<__bf16, 64>(a, n_rows, s) : rows_fwd_g<__bf16, 128>(a, n_rows, s);
}

// ---------------------------------------------------------------- backward
//
// The backward of hga_attend_rows_fwd with the routing held constant, in
// three launches:
//   rows_rowdot_kernel  D = rowsum(dO * O) of every (row, query head);
//   dQ                  query-major: one workgroup per (row, kv head) walks
//                       the row's routed set in 64-key tiles, recomputes P
//                       from the LSE, forms dS = P (dP - D) and accumulates
//                       dQ = scale dS K (rows_dq_mfma_kernel for bf16 on the
//                       matrix cores, rows_dq_kernel for float32);
//   dK, dV              key-major and deterministic: one workgroup per (16
//                       keys of a 64-token chunk of the active tokens, kv
//                       head). It lists, in row order, the rows whose routed
//                       set touches those keys (window or selected groups)
//                       with the mask of the keys each attends, then walks the
//                       list (rows_dkv_mfma_kernel for bf16, rows_dkv_kernel
//                       for float32). No atomics: results are bitwise
//                       reproducible.

template <typename T, int D>
__global__ __launch_bounds__(256) void rows_rowdot_kernel(AttnArgs a, int64_t n_rows) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E = D / 64;
  const int lane = threadIdx.x & 63;
  const int64_t x = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (row, query head)
  if (x >= n_rows * a.n_q_heads) return;
  const int64_t row = x / a.n_q_heads;
  const int hq = (int)(x % a.n_q_heads);
  const char* dob = static_cast<const char*>(a.dO) + (row * a.do_tok + (int64_t)hq * a.do_head) * EB;
  float acc = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int d = lane * E + e;
    const float o = a.o32 ? a.o32[(row * a.n_q_heads + hq) * D + d]
                          : load_elem<T, D>(static_cast<const char*>(a.O) +
                                            (row * a.o_tok + (int64_t)hq * a.o_head + d) * EB);
    acc = fmaf(load_elem<T, D>(dob + (int64_t)d * EB), o, acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) a.dvec[x] = acc;
}

// float32 dQ on the vector units: the four waves stage each tile's K and V
// rows together in LDS (double-buffered); each wave takes a query head,
// forms dS (lane = key), then dQ = scale dS K (lane = head-dim slice, keys in
// tile order).
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void rows_dq_kernel(AttnArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E = D / 64;             // dQ dims of a lane
  constexpr int NP = D * EB / 16;       // 16-byte pieces of a key row
  constexpr int EP = 16 / EB;           // elements per piece
  constexpr int KP = D * EB + 16;       // LDS pitch of a staged K / V row (padded against bank conflicts)
  constexpr int HPW = (G + 3) / 4;      // query heads of a wave
  constexpr int PER = 2 * 64 * NP / 256;  // 16-byte pieces of a K/V tile per thread
  __shared__ __attribute__((aligned(16))) float s_q[G][D];
  __shared__ __attribute__((aligned(16))) float s_do[G][D];
  __shared__ float s_lse[G], s_dd[G];
  __shared__ float s_ds[G][64];
  // the K and V rows of the current 64-key tile, double-buffered
  __shared__ __attribute__((aligned(16))) char s_kv[2][2][64 * KP];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t row = blockIdx.x / a.n_kv_heads;
  const char* Kb = static_cast<const char*>(a.K);
  const char* Vb = static_cast<const char*>(a.V);
  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, e = x % D;
    const int64_t hq = h * G + g;
    s_q[g][e] = load_elem<T, D>(static_cast<const char*>(a.Q) + (row * a.q_tok + hq * a.q_head + e) * EB);
    s_do[g][e] = load_elem<T, D>(static_cast<const char*>(a.dO) + (row * a.do_tok + hq * a.do_head + e) * EB);
  }
  if (tid < G) {
    s_lse[tid] = a.lse[row * a.n_q_heads + h * G + tid] * kLog2e;
    s_dd[tid] = a.dvec[row * a.n_q_heads + h * G + tid];
  }
  const RowSet rs = row_set(a, row, h);
  const int ntiles = (rs.R + 63) / 64;

  // a tile's K and V rows: thread items (tensor, row, piece), all loads in
  // flight together, then stored to the tile's buffer
  const int64_t k_stride = a.k_tok * EB, v_stride = a.v_tok * EB;
  const int64_t k_head = (int64_t)h * a.k_head * EB, v_head = (int64_t)h * a.v_head * EB;
  auto fetch = [&](int tile, u32x4 (&st)[PER]) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int item = tid + 256 * u;
      const int which = item / (64 * NP), rem = item % (64 * NP);
      const int r = rem / NP, c = rem % NP;
      const int p = min(tile * 64 + r, rs.R - 1);  // padding positions read the last row (their P is 0)
      const int64_t t = row_token(p, rs.n_sink, rs.n_grp_tok, rs.ls, rs.sel, a.group_shift);
      const char* src = which == 0 ? row_ptr(Kb, t, k_stride) + k_head : row_ptr(Vb, t, v_stride) + v_head;
      st[u] = *reinterpret_cast<const u32x4*>(src + 16 * c);
    }
  };
  auto stage = [&](int buf, const u32x4 (&st)[PER]) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int item = tid + 256 * u;
      const int which = item / (64 * NP), rem = item % (64 * NP);
      const int r = rem / NP, c = rem % NP;
      *reinterpret_cast<u32x4*>(s_kv[buf][which] + r * KP + 16 * c) = st[u];
    }
  };
  if (ntiles > 0) {
    u32x4 st[PER];
    fetch(0, st);
    stage(0, st);
  }
  __syncthreads();

  float dq[HPW][E];
#pragma unroll
  for (int i = 0; i < HPW; ++i)
#pragma unroll
    for (int e = 0; e < E; ++e) dq[i][e] = 0.0f;
  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    u32x4 nx[PER];
    if (tile + 1 < ntiles) fetch(tile + 1, nx);  // the next tile's rows are in flight during this one
    const char* sk = s_kv[buf][0];
    const char* sv = s_kv[buf][1];
    const int nk = min(64, rs.R - tile * 64);
    // S and dP: lane = key, this wave's query heads
#pragma unroll
    for (int i = 0; i < HPW; ++i) {
      const int g = wave + 4 * i;
      if (g < G) {
        float sg = 0.0f, dg = 0.0f;
#pragma unroll 4
        for (int c = 0; c < NP; ++c) {
          const u32x4 kw = *reinterpret_cast<const u32x4*>(sk + lane * KP + 16 * c);
          const u32x4 vw = *reinterpret_cast<const u32x4*>(sv + lane * KP + 16 * c);
          float kx[EP], vx[EP];
#pragma unroll
          for (int e = 0; e < EP; ++e) {
            if constexpr (EB == 2) {
              kx[e] = bf16_bits_to_float((kw[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
              vx[e] = bf16_bits_to_float((vw[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
            } else {
              kx[e] = __uint_as_float(kw[e]);
              vx[e] = __uint_as_float(vw[e]);
            }
          }
#pragma unroll
          for (int e4 = 0; e4 < EP / 4; ++e4) {
            const f32x4 qq = *reinterpret_cast<const f32x4*>(&s_q[g][c * EP + 4 * e4]);
            const f32x4 dd = *reinterpret_cast<const f32x4*>(&s_do[g][c * EP + 4 * e4]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              sg = fmaf(qq[e], kx[4 * e4 + e], sg);
              dg = fmaf(dd[e], vx[4 * e4 + e], dg);
            }
          }
        }
        const float pr = lane < nk ? exp2f(sg * a.scale_log2 - s_lse[g]) : 0.0f;
        s_ds[g][lane] = pr * (dg - s_dd[g]);
      }
    }
    __builtin_amdgcn_wave_barrier();  // a wave reads only the dS rows it wrote
    // dQ += dS K: lane = head-dim slice, keys of the tile in order
#pragma unroll
    for (int i = 0; i < HPW; ++i) {
      const int g = wave + 4 * i;
      if (g < G) {
#pragma unroll 8
        for (int j = 0; j < nk; ++j) {
          const float dj = s_ds[g][j];
#pragma unroll
          for (int e = 0; e < E; ++e) dq[i][e] = fmaf(dj, load_elem<T, D>(sk + j * KP + (lane * E + e) * EB), dq[i][e]);
        }
      }
    }
    if (tile + 1 < ntiles) {
      // the other buffer held tile - 1, which every wave finished before the
      // previous barrier
      stage(buf ^ 1, nx);
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < HPW; ++i) {
    const int g = wave + 4 * i;
    if (g < G) {
#pragma unroll
      for (int e = 0; e < E; ++e) a.dQ[(row * a.n_q_heads + h * G + g) * D + lane * E + e] = dq[i][e] * a.scale;
    }
  }
}

// bf16: dQ on the matrix cores with the forward's 4x4x4 products. S = Q K^T
// and dP = dO V^T take the heads as the rows of A and lane = key as the
// block column (its own K and V rows), so lane = key receives both for four
// heads; dS = P (dP - D) goes to LDS as a bf16 hi + lo pair (as in the
// block kernels), and dQ += dS K takes the tile's keys as the k axis with K
// read from LDS through the transpose load. Each wave takes every fourth
// 64-key tile; the four partial dQ are added in wave order at the end.
template <int D, int G>
__global__ __launch_bounds__(256) void rows_dq_mfma_kernel(AttnArgs a) {
  constexpr int NG = (G + 3) / 4;  // four-head row groups of A
  constexpr int GR = 4 * NG;       // rows of A (heads past G are zero)
  constexpr int NP = D * 2 / 16;   // 16-byte pieces of a key row
  constexpr int NKS = D / 4;       // k steps of S and dP
  constexpr int NDH = D / 64;      // 64-column slices of dQ
  constexpr int VP = D * 2 + 16;   // LDS pitch of a staged K row (padded against bank conflicts)
  __shared__ __attribute__((aligned(16))) uint16_t s_q[GR][D];        // bf16 query rows of the G heads
  __shared__ __attribute__((aligned(16))) uint16_t s_do[GR][D];       // bf16 dO rows of the G heads
  // each wave's dS as a bf16 hi + lo pair, [head][key]
  __shared__ __attribute__((aligned(16))) uint16_t s_ds[4][GR][64], s_dl[4][GR][64];
  __shared__ float s_lse[G], s_dd[G];
  // each wave's current K tile, row = key; after the tiles, its partial dQ
  __shared__ __attribute__((aligned(16))) char s_k[4][64 * VP];
  static_assert(G * D * 4 <= 64 * VP, "a wave's partial dQ fits its K buffer");
  typedef __attribute__((address_space(3))) s16x4* lds_s4;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t row = blockIdx.x / a.n_kv_heads;
  const char* Kb = static_cast<const char*>(a.K);
  const char* Vb = static_cast<const char*>(a.V);

  for (int x = tid; x < GR * D; x += 256) {
    const int g = x / D, e = x % D;
    const int64_t hq = h * G + g;
    s_q[g][e] = g < G ? *reinterpret_cast<const uint16_t*>(static_cast<const char*>(a.Q) + (row * a.q_tok + hq * a.q_head + e) * 2)
                      : (uint16_t)0;
    s_do[g][e] = g < G ? *reinterpret_cast<const uint16_t*>(static_cast<const char*>(a.dO) + (row * a.do_tok + hq * a.do_head + e) * 2)
                       : (uint16_t)0;
  }
  if constexpr (GR > G) {
    for (int x = tid; x < 4 * (GR - G) * 64; x += 256)
      s_ds[x / ((GR - G) * 64)][G + (x / 64) % (GR - G)][x % 64] = s_dl[x / ((GR - G) * 64)][G + (x / 64) % (GR - G)][x % 64] = 0;
  }
  if (tid < G) {
    s_lse[tid] = a.lse[row * a.n_q_heads + h * G + tid] * kLog2e;
    s_dd[tid] = a.dvec[row * a.n_q_heads + h * G + tid];
  }
  const RowSet rs = row_set(a, row, h);
  __syncthreads();

  f32x4 dq[NG][NDH];
#pragma unroll
  for (int ng = 0; ng < NG; ++ng)
#pragma unroll
    for (int dh = 0; dh < NDH; ++dh) dq[ng][dh] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  const int64_t k_stride = a.k_tok * 2, v_stride = a.v_tok * 2;
  const int64_t k_head = (int64_t)h * a.k_head * 2, v_head = (int64_t)h * a.v_head * 2;
  char* sk = s_k[wave];
  uint16_t(*sds)[64] = s_ds[wave];
  uint16_t(*sdl)[64] = s_dl[wave];
  for (int tb = wave * 64; tb < rs.R; tb += 256) {
    const int p = tb + lane;
    const bool valid = p < rs.R;
    const int64_t t = row_token(min(p, rs.R - 1), rs.n_sink, rs.n_grp_tok, rs.ls, rs.sel, a.group_shift);
    const char* kr = row_ptr(Kb, t, k_stride) + k_head;
    const char* vrow = row_ptr(Vb, t, v_stride) + v_head;
    u32x4 kw[NP], vw[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) kw[c] = *reinterpret_cast<const u32x4*>(kr + 16 * c);
#pragma unroll
    for (int c = 0; c < NP; ++c) vw[c] = *reinterpret_cast<const u32x4*>(vrow + 16 * c);
    // S and dP: this lane's key against the G heads, four heads per product
    f32x4 sacc[NG], pacc[NG];
#pragma unroll
    for (int ng = 0; ng < NG; ++ng) sacc[ng] = pacc[ng] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const u32x4 kc = kw[ks / 2], vc = vw[ks / 2];
      const s16x4 kb = __builtin_bit_cast(s16x4, uint2{kc[2 * (ks % 2)], kc[2 * (ks % 2) + 1]});
      const s16x4 vb = __builtin_bit_cast(s16x4, uint2{vc[2 * (ks % 2)], vc[2 * (ks % 2) + 1]});
#pragma unroll
      for (int ng = 0; ng < NG; ++ng) {
        const s16x4 qa = *reinterpret_cast<const s16x4*>(&s_q[4 * ng + (lane & 3)][4 * ks]);
        const s16x4 da = *reinterpret_cast<const s16x4*>(&s_do[4 * ng + (lane & 3)][4 * ks]);
        sacc[ng] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(qa, kb, sacc[ng], 0, 0, 0);
        pacc[ng] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(da, vb, pacc[ng], 0, 0, 0);
      }
    }
    // dS = P (dP - D), P recomputed from the LSE; dQ multiplies dS by raw
    // keys, whose magnitude is not bounded, so dS is carried as hi + lo
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float pr = valid ? exp2f(sacc[g / 4][g % 4] * a.scale_log2 - s_lse[g]) : 0.0f;
      const float ds = pr * (pacc[g / 4][g % 4] - s_dd[g]);
      const uint32_t hi = float_to_bf16_bits(ds);
      sds[g][lane] = (uint16_t)hi;
      sdl[g][lane] = (uint16_t)float_to_bf16_bits(ds - bf16_bits_to_float(hi));
    }
#pragma unroll
    for (int c = 0; c < NP; ++c) *reinterpret_cast<u32x4*>(sk + lane * VP + 16 * c) = kw[c];
    __builtin_amdgcn_wave_barrier();
    // dQ += dS K over the tile's 64 keys, four keys per k step
    const int i = lane & 15, col0 = 16 * (lane >> 4) + 4 * (i & 3);
#pragma unroll 4
    for (int kk = 0; kk < 16; ++kk) {
      s16x4 da[NG], dl[NG];
#pragma unroll
      for (int ng = 0; ng < NG; ++ng) {
        da[ng] = *reinterpret_cast<const s16x4*>(&sds[4 * ng + (lane & 3)][4 * kk]);
        dl[ng] = *reinterpret_cast<const s16x4*>(&sdl[4 * ng + (lane & 3)][4 * kk]);
      }
#pragma unroll
      for (int dh = 0; dh < NDH; ++dh) {
        const s16x4 kb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s4)(sk + (4 * kk + (i >> 2)) * VP + (64 * dh + col0) * 2));
#pragma unroll
        for (int ng = 0; ng < NG; ++ng) {
          dq[ng][dh] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(da[ng], kb, dq[ng][dh], 0, 0, 0);
          dq[ng][dh] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(dl[ng], kb, dq[ng][dh], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  // the four waves' partial dQ, each in its own K buffer, added in wave order
  float* so = reinterpret_cast<float*>(sk);
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int dh = 0; dh < NDH; ++dh) so[g * D + 64 * dh + lane] = dq[g / 4][dh][g % 4];
  __syncthreads();
  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, e = x % D;
    float acc = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) acc += reinterpret_cast<const float*>(s_k[w])[g * D + e];
    a.dQ[(row * a.n_q_heads + h * G + g) * D + e] = acc * a.scale;
  }
}

// The rows of the call whose routed set touches keys [k0, k0 + KW) of chunk c
// (k0 = 64 c + part KW): listed in row order in s_rows, each with the mask of
// those keys it attends (window or selected groups, cut at its position) in
// s_mask; returns their number. Called by all 256 threads of a workgroup.
template <int KW>
__device__ inline int rows_attending(const AttnArgs& a, int64_t n_rows, int h, int64_t c, int part, int* s_rows,
                                     uint32_t* s_mask, int* s_cnt) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t c0 = c * 64;
  const int64_t k0 = c0 + part * KW;
  const int g_sz = 1 << a.group_shift;
  const int gpc_shift = 6 - a.group_shift;
  const uint64_t kmask = (1ull << KW) - 1;
  int base = 0;
  for (int64_t r0 = 0; r0 < n_rows; r0 += 256) {
    const int64_t r = r0 + tid;
    uint64_t m = 0;
    if (r < n_rows) {
      const int64_t pos = a.q_begin + r;
      if (pos >= k0) {
        const int64_t block_end = (pos / 64 + 1) * 64;
        const int64_t ls = block_end - a.local_tokens > 0 ? block_end - a.local_tokens : 0;
        const int64_t sink_end = min((int64_t)a.sink_tokens, ls);
        if ((c0 >= ls && c0 < block_end) || c0 < sink_end) {
          m = ~0ull;
        } else if (a.top_groups > 0) {
          const int64_t slot = r * a.n_kv_heads + h;
          const int n = a.n_sel[slot];
          const int32_t* sel = a.sel_groups + slot * a.top_groups;
          const uint64_t gm = g_sz == 64 ? ~0ull : (1ull << g_sz) - 1;
          for (int j = 0; j < n; ++j) {
            const int gid = sel[j];
            if ((gid >> gpc_shift) == c) m |= gm << ((gid & ((1 << gpc_shift) - 1)) << a.group_shift);
          }
        }
        const int64_t last = pos - c0;  // keys after the row are not attended
        if (last < 63) m &= (2ull << last) - 1;
        m = (m >> (part * KW)) & kmask;
      }
    }
    const uint64_t bal = __ballot(m != 0);
    if (lane == 0) s_cnt[wave] = __popcll(bal);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wave; ++w) off += s_cnt[w];
    if (m != 0) {
      const int at = off + lanes_below(bal);
      s_rows[at] = (int)r;
      s_mask[at] = (uint32_t)m;
    }
    base += s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    __syncthreads();
  }
  return base;
}

// float32 dK and dV on the vector units: the list is walked four rows at a
// time; the waves split the (row, query head) pairs for S and dP (lane = key
// and a quarter of the head dim, quarters added across lanes), share P and dS
// through LDS, and each thread accumulates a slice of dK and dV for one key.
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void rows_dkv_kernel(AttnArgs a, int64_t n_rows) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int KW = kRowsDkvKeys;     // keys of this workgroup
  constexpr int NQ = 64 / KW;          // lanes per key: head-dim parts of a dot product
  constexpr int DQ = D / NQ;           // head dims of one part
  constexpr int NPQ = DQ * EB / 16;    // 16-byte pieces of one part of a row
  constexpr int EP = 16 / EB;
  constexpr int DE = DQ / 4;           // dK / dV dims a thread accumulates
  __shared__ int s_rows[kRowsBwdMaxRows];  // the row lists live in LDS: calls of at most this many rows
  __shared__ uint32_t s_mask[kRowsBwdMaxRows];
  __shared__ int s_cnt[4];
  constexpr int RB = 4;                // listed rows per step
  __shared__ __attribute__((aligned(16))) float s_q[2][RB][G][D];
  __shared__ __attribute__((aligned(16))) float s_do[2][RB][G][D];
  __shared__ float s_lse[2][RB][G], s_dd[2][RB][G];
  __shared__ float s_p[RB][G][KW], s_ds[RB][G][KW];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int part = (blockIdx.x / a.n_kv_heads) % (64 / KW);
  const int64_t c = a.grad_begin / 64 + blockIdx.x / a.n_kv_heads / (64 / KW);  // absolute chunk
  const int64_t k0 = c * 64 + part * KW;  // this workgroup's first key
  const int64_t q_end = a.q_begin + n_rows;

  // ---- the rows that attend one of this workgroup's keys, in row order,
  // with the mask of those keys each attends
  const int L = rows_attending<KW>(a, n_rows, h, c, part, s_rows, s_mask, s_cnt);

  // ---- this lane's key and head-dim part for the dot products
  const int kk = lane % KW, qd = lane / KW;
  const int64_t tk = min(k0 + kk, q_end - 1);  // keys past the call's end are never attended
  const char* kr = row_ptr(static_cast<const char*>(a.K), tk, a.k_tok * EB) + ((int64_t)h * a.k_head + qd * DQ) * EB;
  const char* vr = row_ptr(static_cast<const char*>(a.V), tk, a.v_tok * EB) + ((int64_t)h * a.v_head + qd * DQ) * EB;
  u32x4 kw[NPQ], vw[NPQ];
#pragma unroll
  for (int p = 0; p < NPQ; ++p) kw[p] = *reinterpret_cast<const u32x4*>(kr + 16 * p);
#pragma unroll
  for (int p = 0; p < NPQ; ++p) vw[p] = *reinterpret_cast<const u32x4*>(vr + 16 * p);
  // this thread's dK / dV dims: key kk, dims [dd0, dd0 + DE)
  const int dd0 = qd * DQ + wave * DE;
  float dk[DE], dv[DE];
#pragma unroll
  for (int e = 0; e < DE; ++e) dk[e] = dv[e] = 0.0f;

  // The list is walked RB rows at a time: the query-side data of the RB
  // rows (all G heads) is staged in LDS, double-buffered, with the next
  // batch's loads in flight while this one is used.
  constexpr int NV = 2 * RB * G * D;            // staged values per batch (Q and dO rows)
  constexpr int PER = (NV + 255) / 256;         // values per thread
  auto fetch = [&](int kb, float (&st)[PER]) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int x = tid + 256 * u;
      const int which = x / (RB * G * D), rem = x % (RB * G * D);
      const int r = rem / (G * D), g = (rem / D) % G, e = rem % D;
      const int64_t rr = s_rows[min(kb + r, L - 1)];
      const int64_t hq = h * G + g;
      st[u] = 0.0f;
      if (x < NV)
        st[u] = which == 0
            ? load_elem<T, D>(static_cast<const char*>(a.Q) + (rr * a.q_tok + hq * a.q_head + e) * EB)
            : load_elem<T, D>(static_cast<const char*>(a.dO) + (rr * a.do_tok + hq * a.do_head + e) * EB);
    }
  };
  auto stage = [&](int kb, int buf, const float (&st)[PER]) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int x = tid + 256 * u;
      const int which = x / (RB * G * D), rem = x % (RB * G * D);
      const int r = rem / (G * D), g = (rem / D) % G, e = rem % D;
      if (x < NV) {
        if (which == 0) s_q[buf][r][g][e] = st[u];
        else s_do[buf][r][g][e] = st[u];
      }
    }
    if (tid < RB * G) {
      const int r = tid / G, g = tid % G;
      const int64_t rr = s_rows[min(kb + r, L - 1)];
      s_lse[buf][r][g] = a.lse[rr * a.n_q_heads + h * G + g] * kLog2e;
      s_dd[buf][r][g] = a.dvec[rr * a.n_q_heads + h * G + g];
    }
  };
  if (L > 0) {
    float st[PER];
    fetch(0, st);
    stage(0, 0, st);
  }
  __syncthreads();
  for (int kb = 0; kb < L; kb += RB) {
    const int buf = (kb / RB) & 1;
    const int nrb = min(RB, L - kb);
    float nx[PER];
    fetch(kb + RB, nx);  // the next batch's data is in flight during this one
    // S and dP of the batch's (row, head) pairs, split over the waves: lane =
    // (key, head-dim part); the NQ parts are added across lanes in a fixed
    // order, so every lane of a key holds the same sums
#pragma unroll 1
    for (int pi = wave; pi < RB * G; pi += 4) {
      const int r = pi / G, g = pi % G;
      if (r < nrb) {
        float s = 0.0f, dp = 0.0f;
#pragma unroll
        for (int p = 0; p < NPQ; ++p) {
          float kx[EP], vx[EP];
#pragma unroll
          for (int e = 0; e < EP; ++e) {
            if constexpr (EB == 2) {
              kx[e] = bf16_bits_to_float((kw[p][e >> 1] >> ((e & 1) * 16)) & 0xffffu);
              vx[e] = bf16_bits_to_float((vw[p][e >> 1] >> ((e & 1) * 16)) & 0xffffu);
            } else {
              kx[e] = __uint_as_float(kw[p][e]);
              vx[e] = __uint_as_float(vw[p][e]);
            }
          }
#pragma unroll
          for (int e4 = 0; e4 < EP / 4; ++e4) {
            const f32x4 qq = *reinterpret_cast<const f32x4*>(&s_q[buf][r][g][qd * DQ + p * EP + 4 * e4]);
            const f32x4 dd = *reinterpret_cast<const f32x4*>(&s_do[buf][r][g][qd * DQ + p * EP + 4 * e4]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              s = fmaf(qq[e], kx[4 * e4 + e], s);
              dp = fmaf(dd[e], vx[4 * e4 + e], dp);
            }
          }
        }
#pragma unroll
        for (int m = KW; m < 64; m <<= 1) {
          s += __shfl_xor(s, m);
          dp += __shfl_xor(dp, m);
        }
        if (qd == 0) {
          const bool attend = (s_mask[kb + r] >> kk) & 1u;
          const float pr = attend ? exp2f(s * a.scale_log2 - s_lse[buf][r][g]) : 0.0f;
          s_p[r][g][kk] = pr;
          s_ds[r][g][kk] = pr * (dp - s_dd[buf][r][g]);
        }
      }
    }
    __syncthreads();
    // dV += P^T dO and dK += dS^T Q: key kk, dims [dd0, dd0 + DE)
#pragma unroll 1
    for (int pi = 0; pi < nrb * G; ++pi) {
      const int r = pi / G, g = pi % G;
      const float pj = s_p[r][g][kk], dj = s_ds[r][g][kk];
#pragma unroll
      for (int e4 = 0; e4 < DE / 4; ++e4) {
        const f32x4 dd = *reinterpret_cast<const f32x4*>(&s_do[buf][r][g][dd0 + 4 * e4]);
        const f32x4 qq = *reinterpret_cast<const f32x4*>(&s_q[buf][r][g][dd0 + 4 * e4]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dv[4 * e4 + e] = fmaf(pj, dd[e], dv[4 * e4 + e]);
          dk[4 * e4 + e] = fmaf(dj, qq[e], dk[4 * e4 + e]);
        }
      }
    }
    if (kb + RB < L) stage(kb + RB, buf ^ 1, nx);
    __syncthreads();
  }
  // keys of this workgroup that exist in this call (all tokens >= grad_begin)
  const int64_t t = k0 + kk;
  if (t < q_end) {
    float* dkr = a.dK + ((t - a.grad_begin) * a.n_kv_heads + h) * D + dd0;
    float* dvr = a.dV + ((t - a.grad_begin) * a.n_kv_heads + h) * D + dd0;
#pragma unroll
    for (int e4 = 0; e4 < DE / 4; ++e4) {
      *reinterpret_cast<f32x4*>(dkr + 4 * e4) =
          f32x4{dk[4 * e4] * a.scale, dk[4 * e4 + 1] * a.scale, dk[4 * e4 + 2] * a.scale, dk[4 * e4 + 3] * a.scale};
      *reinterpret_cast<f32x4*>(dvr + 4 * e4) = f32x4{dv[4 * e4], dv[4 * e4 + 1], dv[4 * e4 + 2], dv[4 * e4 + 3]};
    }
  }
}

// bf16: dK and dV on the matrix cores. The waves take every fourth batch of
// 16 (row, query head) pairs of the list (16 / G rows each). S = Q K^T and
// dP = dO V^T are 16 x 16 x d products (v_mfma_f32_16x16x32_bf16, lane l
// holding row l % 16 of A and column l % 16 of B over eight k values):
// A = the batch's Q or dO rows, B = the workgroup's 16 K or V rows, held in
// registers for the whole walk. Their result holds, in lane l, pairs
// 4 (l / 16) .. + 3 of key l % 16, which is the A operand of the 16 x 16 x 16
// product with keys as rows: P and dS, each as a bf16 hi + lo pair (two
// products sharing the B operand, so both enter to about 2^-17), feed
// dV += P^T dO and dK += dS^T Q straight from the registers, with dO and Q
// read from LDS through the transpose load. Each wave keeps its own dK and
// dV; the four are added in wave order at the end, so results are bitwise
// reproducible.
template <int D, int G>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void rows_dkv_mfma_kernel(AttnArgs a,
                                                                                     int64_t n_rows) {
  constexpr int KW = kRowsDkvKeys;  // keys of this workgroup
  static_assert(KW == 16, "one 16 x 16 product per batch");
  constexpr int PR = 16 / G;        // rows of a batch
  constexpr int NS = D / 32;        // k steps of S and dP
  constexpr int NT = D / 16;        // 16-column tiles of dK and dV
  constexpr int QP = D * 2 + 16;    // LDS pitch of a staged Q / dO row (padded against bank conflicts)
  __shared__ int s_rows[kRowsBwdMaxRows];  // the row lists live in LDS: calls of at most this many rows
  __shared__ uint32_t s_mask[kRowsBwdMaxRows];
  __shared__ int s_cnt[4];
  // each wave's Q and dO rows of its current batch; at the end, its partial dV, then dK
  __shared__ __attribute__((aligned(16))) char s_st[4][2][16 * QP];
  static_assert(KW * D * 4 <= 2 * 16 * QP, "a wave's partial dK or dV fits its staging buffer");
  typedef __attribute__((address_space(3))) s16x4* lds_s4;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int part = (blockIdx.x / a.n_kv_heads) % (64 / KW);
  const int64_t c = a.grad_begin / 64 + blockIdx.x / a.n_kv_heads / (64 / KW);  // absolute chunk
  const int64_t k0 = c * 64 + part * KW;  // this workgroup's first key
  const int64_t q_end = a.q_begin + n_rows;

  const int L = rows_attending<KW>(a, n_rows, h, c, part, s_rows, s_mask, s_cnt);

  // lane l: key kk of the workgroup (B column of S and dP, pair row of their
  // A), and quad, which selects the eight-value k slices it holds
  const int kk = lane & 15, quad = lane >> 4;
  const int64_t tk = min(k0 + kk, q_end - 1);  // keys past the call's end are never attended
  const char* kr = row_ptr(static_cast<const char*>(a.K), tk, a.k_tok * 2) + (int64_t)h * a.k_head * 2;
  const char* vr = row_ptr(static_cast<const char*>(a.V), tk, a.v_tok * 2) + (int64_t)h * a.v_head * 2;
  u32x4 kb[NS], vb[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    kb[s] = *reinterpret_cast<const u32x4*>(kr + (4 * s + quad) * 16);
    vb[s] = *reinterpret_cast<const u32x4*>(vr + (4 * s + quad) * 16);
  }
  f32x4 dk[NT], dv[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dk[t] = dv[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  // a batch's operands: this lane's A slices (pair kk) and the softmax data of
  // its four result pairs 4 quad + i; entries past the list repeat its last
  // row and attend nothing
  struct Batch {
    u32x4 q[NS], d[NS];
    float lse[4], dd[4];
    uint32_t att;
  };
  auto fetch = [&](int kb0, Batch& b) {
    const int64_t ra = s_rows[min(kb0 + kk / G, L - 1)];
    const int64_t hqa = (int64_t)h * G + kk % G;
    const char* qr = static_cast<const char*>(a.Q) + (ra * a.q_tok + hqa * a.q_head) * 2;
    const char* dr = static_cast<const char*>(a.dO) + (ra * a.do_tok + hqa * a.do_head) * 2;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      b.q[s] = *reinterpret_cast<const u32x4*>(qr + (4 * s + quad) * 16);
      b.d[s] = *reinterpret_cast<const u32x4*>(dr + (4 * s + quad) * 16);
    }
    b.att = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = 4 * quad + i, e = kb0 + p / G, ec = min(e, L - 1);
      const int64_t x = (int64_t)s_rows[ec] * a.n_q_heads + h * G + p % G;
      b.lse[i] = a.lse[x] * kLog2e;
      b.dd[i] = a.dvec[x];
      if (e < L && ((s_mask[ec] >> kk) & 1u)) b.att |= 1u << i;
    }
  };
  char* sq = s_st[wave][0];
  char* sdo = s_st[wave][1];
  const int rd = (4 * quad + (kk >> 2)) * QP + 4 * (kk & 3) * 2;  // this lane's transpose-load address in a tile
  Batch cur;
  if (wave * PR < L) fetch(wave * PR, cur);
  for (int kb0 = wave * PR; kb0 < L; kb0 += 4 * PR) {
    Batch nxt;
    if (kb0 + 4 * PR < L) fetch(kb0 + 4 * PR, nxt);  // the next batch's loads are in flight during this one
    f32x4 sacc = {0.0f, 0.0f, 0.0f, 0.0f}, pacc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, cur.q[s]),
                                                     __builtin_bit_cast(bf16x8, kb[s]), sacc, 0, 0, 0);
      pacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, cur.d[s]),
                                                     __builtin_bit_cast(bf16x8, vb[s]), pacc, 0, 0, 0);
    }
    // the batch's Q and dO rows into this wave's staging tiles (row = pair)
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      *reinterpret_cast<u32x4*>(sq + kk * QP + (4 * s + quad) * 16) = cur.q[s];
      *reinterpret_cast<u32x4*>(sdo + kk * QP + (4 * s + quad) * 16) = cur.d[s];
    }
    // P and dS = P (dP - D) of pairs 4 quad + i against key kk
    s16x4 pa, pl, sa, sl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pr = (cur.att >> i) & 1u ? exp2f(sacc[i] * a.scale_log2 - cur.lse[i]) : 0.0f;
      const float ds = pr * (pacc[i] - cur.dd[i]);
      const uint32_t ph = float_to_bf16_bits(pr), dh = float_to_bf16_bits(ds);
      pa[i] = (short)ph;
      pl[i] = (short)float_to_bf16_bits(pr - bf16_bits_to_float(ph));
      sa[i] = (short)dh;
      sl[i] = (short)float_to_bf16_bits(ds - bf16_bits_to_float(dh));
    }
    __builtin_amdgcn_wave_barrier();
    // dV += P^T dO and dK += dS^T Q, sixteen columns per product
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const s16x4 bo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(sdo + rd + 32 * t));
      const s16x4 bq = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(sq + rd + 32 * t));
      dv[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, bo, dv[t], 0, 0, 0);
      dv[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl, bo, dv[t], 0, 0, 0);
      dk[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sa, bq, dk[t], 0, 0, 0);
      dk[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(sl, bq, dk[t], 0, 0, 0);
    }
    __builtin_amdgcn_wave_barrier();
    cur = nxt;
  }
  // the four waves' partial dV, then dK, added in wave order; lane l holds
  // keys 4 quad + i, column 16 t + kk
  __syncthreads();
  for (int which = 0; which < 2; ++which) {
    float* pd = reinterpret_cast<float*>(s_st[wave]);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) pd[(4 * quad + i) * D + 16 * t + kk] = which == 0 ? dv[t][i] : dk[t][i];
    __syncthreads();
    for (int x = tid; x < KW * D / 4; x += 256) {
      const int key = x / (D / 4), col = 4 * (x % (D / 4));
      f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int w = 0; w < 4; ++w) acc += *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(s_st[w]) + key * D + col);
      const int64_t t = k0 + key;
      if (t < q_end) {  // keys of this workgroup that exist in this call (all tokens >= grad_begin)
        float* dst = (which == 0 ? a.dV : a.dK) + ((t - a.grad_begin) * a.n_kv_heads + h) * D + col;
        *reinterpret_cast<f32x4*>(dst) = which == 0 ? acc : acc * a.scale;
      }
    }
    __syncthreads();
  }
}

template <typename T, int D, int G>
hipError_t rows_bwd_g(const AttnArgs& a, int64_t n_rows, hipStream_t s) {
  const int64_t q_end = a.q_begin + n_rows;
  const int n_act = (int)((q_end - a.grad_begin + 63) / 64);
  if constexpr (Elem<T>::kBytes == 2)
    hipLaunchKernelGGL((rows_dq_mfma_kernel<D, G>), dim3((unsigned)(n_rows * a.n_kv_heads)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((rows_dq_kernel<T, D, G>), dim3((unsigned)(n_rows * a.n_kv_heads)), dim3(256), 0, s, a);
  const dim3 dkv_grid((unsigned)(n_act * a.n_kv_heads * (64 / kRowsDkvKeys)));
  if constexpr (Elem<T>::kBytes == 2)
    hipLaunchKernelGGL((rows_dkv_mfma_kernel<D, G>), dkv_grid, dim3(256), 0, s, a, n_rows);
  else
    hipLaunchKernelGGL((rows_dkv_kernel<T, D, G>), dkv_grid, dim3(256), 0, s, a, n_rows);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t rows_bwd_d(const AttnArgs& a, int64_t n_rows, hipStream_t s) {
  const int64_t pairs = n_rows * a.n_q_heads;
  hipLaunchKernelGGL((rows_rowdot_kernel<T, D>), dim3((unsigned)((pairs + 3) / 4)), dim3(256), 0, s, a, n_rows);
  switch (a.gqa) {
    case 1: return rows_bwd_g<T, D, 1>(a, n_rows, s);
    case 2: return rows_bwd_g<T, D, 2>(a, n_rows, s);
    case 4: return rows_bwd_g<T, D, 4>(a, n_rows, s);
    default: return rows_bwd_g<T, D, 8>(a, n_rows, s);
  }
}

hipError_t launch_attend_rows_bwd(const AttnArgs& a, int64_t n_rows, bool bf16, int head_dim, hipStream_t s) {
  if (!bf16) return rows_bwd_d<float, 64>(a, n_rows, s);  // float32 is built for head_dim 64 only
  return head_dim == 64 ? rows_bwd_d<__bf16, 64>(a, n_rows, s) : rows_bwd_d<__bf16, 128>(a, n_rows, s);
}

}  // namespace hga
