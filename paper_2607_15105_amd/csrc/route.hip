// Two-level routing (Sec. 2.1 items 1-2, Fig. 1): block descriptor, chunk
// scoring + top-k_c, group scoring + top-k_g.
//
// qbar_kernel   one workgroup per (query block, kv head): a bandwidth-bound
//               pass over the block's B x G query rows, summed exactly in
//               float64 (bf16 has 8 significant bits), scaled by 1/(B*G).
// route_kernel  one workgroup per (TB consecutive query blocks, kv head).
//               Phase 1 streams every candidate chunk summary once and scores
//               it against all TB descriptors (lane = chunk; the descriptors
//               are wave-uniform and live in scalar registers), keeping
//               float64 scores in LDS. Phase 2: one wave per block extracts
//               the top-k_c with a cached per-lane top-2 tournament, then
//               sorts the winners ascending with a bitonic network across
//               lanes. Phase 3 repeats scoring and selection over the groups
//               of the chosen chunks. Equal scores keep the lower index.
#include "hga_device.h"
#include "hga_kernels.h"

namespace hga {

// ----------------------------------------------------------------------------
// Block descriptor: qbar[b][h][:] = mean over rows of block b and heads of h.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void qbar_kernel(QbarArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E2 = 16 / EB;
  const int h = blockIdx.x % a.n_kv_heads;
  const int b = blockIdx.x / a.n_kv_heads;
  const int D = a.head_dim;
  const int G = a.gqa;
  const int cpq = G * D / E2;           // 16-byte slices per query row (G heads)
  const int nsub = blockDim.x / cpq;    // rows processed in parallel
  const int col = threadIdx.x % cpq;
  const int sub = threadIdx.x / cpq;
  __shared__ double acc[256 * 8];       // [thread][E2]
  double s[E2];
#pragma unroll
  for (int e = 0; e < E2; ++e) s[e] = 0.0;
  const int gq = (col * E2) / D;
  const int d0 = (col * E2) % D;
  const char* Qb = static_cast<const char*>(a.Q);
  if (sub < nsub) {
    for (int r = sub; r < 64; r += nsub) {
      const int64_t off = ((int64_t)(b * 64 + r) * a.q_tok + (int64_t)(h * G + gq) * a.q_head + d0) * EB;
      const uint4 raw = *reinterpret_cast<const uint4*>(Qb + off);
      const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < E2; ++e) {
        float x;
        if constexpr (EB == 2) x = bf16_bits_to_float((w[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
        else x = __uint_as_float(w[e]);
        s[e] += (double)x;
      }
    }
  }
#pragma unroll
  for (int e = 0; e < E2; ++e) acc[threadIdx.x * 8 + e] = s[e];
  __syncthreads();
  // thread d sums over the row subsets and the G heads of element d
  const double inv = 1.0 / (64.0 * G);
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    double tot = 0.0;
    const int cd = d / E2, ed = d % E2;
    for (int g2 = 0; g2 < G; ++g2) {
      const int c2 = g2 * (D / E2) + cd;
      for (int sb = 0; sb < nsub; ++sb) tot += acc[(sb * cpq + c2) * 8 + ed];
    }
    a.qbar[((int64_t)b * a.n_kv_heads + h) * D + d] = tot * inv;
  }
}

hipError_t launch_qbar(const QbarArgs& a, bool bf16, hipStream_t s) {
  const int E2 = bf16 ? 8 : 4;
  const int cpq = a.gqa * a.head_dim / E2;
  const int threads = cpq >= 256 ? 256 : (256 / cpq) * cpq;
  const dim3 grid(a.n_qb * a.n_kv_heads);
  if (bf16)
    hipLaunchKernelGGL(qbar_kernel<__bf16>, grid, dim3(threads), 0, s, a);
  else
    hipLaunchKernelGGL(qbar_kernel<float>, grid, dim3(threads), 0, s, a);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Selection helpers. Order: larger score first, lower index on equal scores.
// ----------------------------------------------------------------------------
__device__ inline bool better(double va, int ia, double vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__device__ inline double shfl_xor_d(double v, int m) {
  const uint64_t u = __double_as_longlong(v);
  const int lo = __shfl_xor((int)(uint32_t)u, m, 64);
  const int hi = __shfl_xor((int)(uint32_t)(u >> 32), m, 64);
  return __longlong_as_double(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

constexpr int kNoIdx = 0x7fffffff;

// Best two not-yet-taken entries of this lane's strided slice sc[lane + 64 j].
__device__ inline void lane_top2(const double* sc, int n, int lane, double& v1, int& i1,
                                 double& v2, int& i2) {
  v1 = -__builtin_inf(); i1 = kNoIdx; v2 = -__builtin_inf(); i2 = kNoIdx;
  for (int i = lane; i < n; i += 64) {
    const double v = sc[i];
    if (v == -__builtin_inf()) continue;  // taken (scores of finite inputs are finite)
    if (better(v, i, v1, i1)) { v2 = v1; i2 = i1; v1 = v; i1 = i; }
    else if (better(v, i, v2, i2)) { v2 = v; i2 = i; }
  }
}

// Top-k positions of sc[0..n) (k <= 64), returned ascending in lanes [0, k_eff);
// lanes >= k_eff return kNoIdx. Taken entries of sc are overwritten with -inf.
__device__ int wave_top_k(double* sc, int n, int k, int lane) {
  const int k_eff = min(k, n);
  double v1, v2;
  int i1, i2;
  lane_top2(sc, n, lane, v1, i1, v2, i2);
  int mine = kNoIdx;
  for (int r = 0; r < k_eff; ++r) {
    double bv = v1;
    int bi = i1;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const double ov = shfl_xor_d(bv, m);
      const int oi = __shfl_xor(bi, m, 64);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == r) mine = bi;
    bool rescan = false;
    if ((bi & 63) == lane) {  // this lane owned the winner
      sc[bi] = -__builtin_inf();
      v1 = v2; i1 = i2;
      v2 = -__builtin_inf(); i2 = kNoIdx;
      rescan = (i1 == kNoIdx);
    }
    if (__any(rescan)) {
      if (rescan) lane_top2(sc, n, lane, v1, i1, v2, i2);
    }
  }
  // bitonic sort (ascending) of the winners across the 64 lanes
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride >= 1; stride >>= 1) {
      const int other = __shfl_xor(mine, stride, 64);
      const bool up = ((lane & size) == 0);
      const bool lower = ((lane & stride) == 0);
      const int lo = min(mine, other), hi = max(mine, other);
      mine = (lower == up) ? lo : hi;
    }
  }
  return mine;
}

// Score of one summary row (D floats) against a wave-uniform float64 descriptor.
template <int D>
__device__ inline double score_row(const float* row, const double* __restrict__ q) {
  double acc = 0.0;
#pragma unroll 8
  for (int d = 0; d < D; d += 4) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(row + d);
    acc = fma((double)v[0], q[d], acc);
    acc = fma((double)v[1], q[d + 1], acc);
    acc = fma((double)v[2], q[d + 2], acc);
    acc = fma((double)v[3], q[d + 3], acc);
  }
  return acc;
}

// One past the last candidate chunk of absolute query block `blk`: chunks end
// at or before the start of the block's local window.
__device__ inline int last_cand(int64_t blk, int local_tokens) {
  const int64_t ls = (blk + 1) * 64 - local_tokens;
  return ls > 0 ? (int)(ls / 64) : 0;
}

template <int D, int TB>
__global__ __launch_bounds__(256) void route_kernel(RouteArgs a) {
  extern __shared__ double sc_all[];  // [TB][score_stride]
  __shared__ int s_chunks[TB * 64];   // chosen chunks of each block, ascending
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = blockIdx.x % a.n_kv_heads;
  const int b0 = (blockIdx.x / a.n_kv_heads) * TB;
  const int nb = min(TB, a.n_qb - b0);  // blocks handled by this workgroup
  const int64_t qb_abs0 = a.q_begin / 64 + b0;

  // candidate chunk range of block i: [first_cand, last_cand(i))
  const int c_lo = a.first_cand;
  const int c_hi = last_cand(qb_abs0 + nb - 1, a.local_tokens);
  const int n_union = c_hi > c_lo ? c_hi - c_lo : 0;

  // ---- phase 1: chunk scores for all TB blocks (summary rows read once)
  const double* qb[TB];
#pragma unroll
  for (int i = 0; i < TB; ++i) {
    const int bi = min(i, nb - 1);
    qb[i] = a.qbar + ((int64_t)(b0 + bi) * a.n_kv_heads + h) * D;
  }
  const float* cs = a.chunk_sum + (int64_t)h * a.chunk_cap * D;
  for (int i = threadIdx.x; i < n_union; i += blockDim.x) {
    const float* row = cs + (int64_t)(c_lo + i) * D;
    double acc[TB];
#pragma unroll
    for (int t = 0; t < TB; ++t) acc[t] = 0.0;
#pragma unroll 4
    for (int d = 0; d < D; d += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(row + d);
#pragma unroll
      for (int t = 0; t < TB; ++t) {
        acc[t] = fma((double)v[0], qb[t][d], acc[t]);
        acc[t] = fma((double)v[1], qb[t][d + 1], acc[t]);
        acc[t] = fma((double)v[2], qb[t][d + 2], acc[t]);
        acc[t] = fma((double)v[3], qb[t][d + 3], acc[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < TB; ++t) sc_all[t * a.score_stride + i] = acc[t];
  }
  __syncthreads();
  if (wave >= nb) return;

  // ---- phase 2: top-k_c of this wave's block
  const int b = b0 + wave;
  double* sc = sc_all + wave * a.score_stride;
  const int n_cand = max(0, last_cand(qb_abs0 + wave, a.local_tokens) - c_lo);
  const int64_t slot = (int64_t)b * a.n_kv_heads + h;
  const int kc_eff = min(a.top_chunks, n_cand);
  int chunk = kNoIdx;
  if (a.top_chunks > 0) {
    const int pos = wave_top_k(sc, n_cand, a.top_chunks, lane);
    chunk = pos == kNoIdx ? kNoIdx : c_lo + pos;
    if (lane < a.top_chunks)
      a.sel_chunks[slot * a.top_chunks + lane] = lane < kc_eff ? chunk : -1;
  }
  int* my_chunks = s_chunks + wave * 64;
  my_chunks[lane] = chunk;
  __builtin_amdgcn_wave_barrier();

  // ---- phase 3: groups of the chosen chunks, top-k_g
  const int gpc_shift = 6 - a.group_shift;  // log2(groups per chunk)
  const int n_gc = kc_eff << gpc_shift;
  const double* q = a.qbar + slot * D;
  const float* gs = a.group_sum + (int64_t)h * a.group_cap * D;
  for (int i = lane; i < n_gc; i += 64) {
    const int ch = my_chunks[i >> gpc_shift];
    const int64_t j = ((int64_t)ch << gpc_shift) + (i & ((1 << gpc_shift) - 1));
    sc[i] = score_row<D>(gs + j * D, q);
  }
  __builtin_amdgcn_wave_barrier();
  if (a.top_groups > 0) {
    const int kg_eff = min(a.top_groups, n_gc);
    const int pos = wave_top_k(sc, n_gc, a.top_groups, lane);
    if (lane < a.top_groups) {
      int gid = -1;
      if (lane < kg_eff) {
        const int ch = my_chunks[pos >> gpc_shift];
        gid = (ch << gpc_shift) + (pos & ((1 << gpc_shift) - 1));
      }
      a.sel_groups[slot * a.top_groups + lane] = gid;
    }
    if (lane == 0) a.n_sel[slot] = kg_eff;
  } else if (lane == 0) {
    a.n_sel[slot] = 0;
  }
}

hipError_t launch_route(const RouteArgs& a, int head_dim, int tb, size_t lds, hipStream_t s) {
  const dim3 grid(((a.n_qb + tb - 1) / tb) * a.n_kv_heads);
  const dim3 block(64 * tb);
#define HGA_ROUTE(D, TB) hipLaunchKernelGGL((route_kernel<D, TB>), grid, block, lds, s, a)
  if (head_dim == 64) {
    if (tb == 1) HGA_ROUTE(64, 1); else if (tb == 2) HGA_ROUTE(64, 2); else HGA_ROUTE(64, 4);
  } else {
    if (tb == 1) HGA_ROUTE(128, 1); else if (tb == 2) HGA_ROUTE(128, 2); else HGA_ROUTE(128, 4);
  }
#undef HGA_ROUTE
  return hipGetLastError();
}

}  // namespace hga
