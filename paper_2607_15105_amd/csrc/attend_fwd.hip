// Exact-token routed attention, forward (Sec. 2.1 item 3).
//
// One workgroup per (query block, kv head, slice of GW query heads). Each of
// its 2*GW waves owns 32 queries of one query head. The routed key set
// [sink | selected groups | local] is gathered 64 tokens at a time into LDS,
// double-buffered: the next tile's global loads are in flight while the
// matrix cores work on the current one. K and V stay row-major in LDS; the V
// operand of P.V is read with the LDS transpose load (fp32 inputs, which have
// no such load, stage V transposed instead).
//
// Per tile and wave, on 32x32 MFMA tiles:
//   S^T = K . Q^T      (A = K rows from LDS, B = the wave's Q held in registers)
//   online softmax     (every lane holds scores of a single query, so the
//                       running max / sum are per lane plus one cross-half swap)
//   O^T += V^T . P^T   (A = transposed V from LDS, B = P straight from the
//                       S^T accumulators, rounded to the input precision)
// Scores are kept raw; p = exp2(s*c - m*c) with c = softmax_scale*log2(e) is one
// FMA and one v_exp_f32. The running max m is raised lazily: only when a row's
// new maximum exceeds it by more than 2^8 (in exp2 units) are O and the sum
// rescaled, so p stays below 2^8 and most tiles skip the rescale entirely.
#include "route_device.h"
#include "routed_tile.h"

namespace hga {

// The attention of one workgroup: (query block wc.b, kv head wc.h, query heads
// wc.hs * GW ...). `get_rs` yields the block's routed set (it may run the
// routing itself); the query rows and, when tile 0 is all sink, that tile's
// K/V rows are requested before it is called.
// PREC (bf16 only, chosen when the caller asks for the float32 copy of O):
// P enters P.V as a bf16 hi + lo pair, so that copy is accurate to ~2^-17
// relative and the backward's row term D = rowsum(dO * O) is exact enough.
template <typename T, int D, int GW, bool PREC, typename GetRS>
__device__ __forceinline__ void attend_block(const AttnArgs& a, const WgCoord wc, char* smem, GetRS&& get_rs) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS;   // MFMAs over the head dim per S tile
  constexpr int NDT = D / 32;   // 32-wide head-dim tiles of O^T
  constexpr int NPS = 64 / KS;  // MFMA k-steps over a 64-key tile in P.V
  constexpr int VPS = 16 / E;
  constexpr int NT = 128 * GW;
  constexpr bool TR = EB == 2;  // V operand through the LDS transpose load
  constexpr int STAGE = TL::kRowBytes + (TR ? TL::kRowBytes : TL::kTBytes);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int hq = wc.h * a.gqa + wc.hs * GW + (wave >> 1);
  const int qoff = (wave & 1) * 32 + l32;  // query offset inside the block
  const int row = wc.b * 64 + qoff;

  const char* Qb = static_cast<const char*>(a.Q);
  const char* Kb = static_cast<const char*>(a.K);
  const char* Vb = static_cast<const char*>(a.V);
  const int64_t k_head_b = (int64_t)wc.h * a.k_head * EB, v_head_b = (int64_t)wc.h * a.v_head * EB;

  Frag qf[NKS];
  {
    const char* qrow = Qb + ((int64_t)row * a.q_tok + (int64_t)hq * a.q_head) * EB;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = EL::load_frag(qrow + (ks * KS + E * hh) * EB);
  }
  KVRegs<T, D, NT> kv0, kv1, kv2;
  const char* kb = Kb + k_head_b;
  const char* vb = Vb + v_head_b;
  const int64_t ktb = a.k_tok * EB, vtb = a.v_tok * EB;
  // a sink-only first tile goes out with the query rows, before the routed
  // set is known
  const bool tile0_sink = sink_fills_tile0(a, wc.b);
  if (tile0_sink) kv0.load_contiguous(kb, ktb, vb, vtb, 0, tid);
  const RoutedSet rs = get_rs();
  const int ntiles = (rs.R + 63) >> 6;
  f32x16 oacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) oacc[dt] = f32x16{};
  float m_run = -__builtin_inff(), l_run = 0.0f;

  const float c = a.scale_log2;
  const float lazy = 8.0f / c;  // raise the max only when it grows by > 2^8 in exp2 units
  // Three register slots rotate so that three tiles' gathers are in flight
  // while one tile is computed; LDS is double-buffered.
  auto put = [&](const KVRegs<T, D, NT>& r, char* dst) {
    r.store_rows(dst, false, tid);
    if constexpr (TR) r.store_rows(dst + TL::kRowBytes, true, tid);
    else r.store_transposed(dst + TL::kRowBytes, true, tid);
  };
  __syncthreads();  // s_sel
  if (!tile0_sink) kv0.load(kb, ktb, vb, vtb, rs, 0, tid);
  if (ntiles > 1) kv1.load(kb, ktb, vb, vtb, rs, 1, tid);
  if (ntiles > 2) kv2.load(kb, ktb, vb, vtb, rs, 2, tid);
  put(kv0, smem);
  if (ntiles > 3) kv0.load(kb, ktb, vb, vtb, rs, 3, tid);
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const char* st = smem + (tile & 1) * STAGE;
    // S^T = K . Q^T : two 32-key tiles, raw scores
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const Frag kf = EL::load_frag(st + TL::row_off(32 * t + l32, ks * KS + E * hh));
        sacc[t] = EL::mma(kf, qf[ks], sacc[t]);
      }
    }
    if (rs.tile_needs_mask(tile * 64, (wave & 1) * 32)) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int p = tile * 64 + 32 * t + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (rs.masked(p, qoff)) sacc[t][v] = -__builtin_inff();
        }
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[t][v]);
    mx = fmaxf(mx, xor32(mx));
    const bool raise = mx > m_run + lazy;  // also true on the first tile (m_run = -inf)
    if (__any(raise)) {
      const float m_new = raise ? mx : m_run;
      const float corr = __builtin_amdgcn_exp2f((m_run - m_new) * c);
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) oacc[dt] *= corr;
    }
    const float mc = m_run * c;
    float psum = 0.0f;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[t][v], c, -mc));
        sacc[t][v] = p;
        psum += p;
      }
    }
    l_run += psum;
    // O^T += V^T . P^T
#pragma unroll
    for (int s = 0; s < NPS; ++s) {
      float pv[E], plo[E];
#pragma unroll
      for (int j = 0; j < E; ++j) {
        pv[j] = sacc[s / VPS][E * (s % VPS) + j];
        if constexpr (PREC) plo[j] = pv[j] - bf16_bits_to_float(float_to_bf16_bits(pv[j]));
      }
      const Frag pf = EL::frag_from(pv);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        Frag vf;
        if constexpr (TR) vf = tr_frag<TL>(st + TL::kRowBytes, 32 * dt, 16 * s + 4 * hh, 16 * s + 8 + 4 * hh, lane);
        else vf = EL::load_frag(st + TL::kRowBytes + TL::t_off(32 * dt + l32, KS * s + E * hh));
        oacc[dt] = EL::mma(vf, pf, oacc[dt]);
        if constexpr (PREC) oacc[dt] = EL::mma(vf, EL::frag_from(plo), oacc[dt]);
      }
    }
    // the slot holding tile+1 goes to LDS, then refills with tile+4
    if (tile + 1 < ntiles) {
      char* nx = smem + ((tile + 1) & 1) * STAGE;
      const int j = tile % 3;
      if (j == 0) {
        put(kv1, nx);
        if (tile + 4 < ntiles) kv1.load(kb, ktb, vb, vtb, rs, tile + 4, tid);
      } else if (j == 1) {
        put(kv2, nx);
        if (tile + 4 < ntiles) kv2.load(kb, ktb, vb, vtb, rs, tile + 4, tid);
      } else {
        put(kv0, nx);
        if (tile + 4 < ntiles) kv0.load(kb, ktb, vb, vtb, rs, tile + 4, tid);
      }
    }
    __syncthreads();
  }

  // epilogue: O = O^T / l, LSE = (m + log2 l) * ln 2
  const float l = l_run + xor32(l_run);
  const float inv = 1.0f / l;
  char* orow = static_cast<char*>(a.Out) + ((int64_t)row * a.out_tok + (int64_t)hq * a.out_head) * EB;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d = 32 * dt + 8 * v4 + 4 * hh;
      const float o0 = oacc[dt][4 * v4] * inv, o1 = oacc[dt][4 * v4 + 1] * inv;
      const float o2 = oacc[dt][4 * v4 + 2] * inv, o3 = oacc[dt][4 * v4 + 3] * inv;
      if (a.o32)
        *reinterpret_cast<f32x4*>(a.o32 + ((int64_t)row * a.n_q_heads + hq) * D + d) = f32x4{o0, o1, o2, o3};
      if constexpr (EB == 2) {
        uint2 w;
        w.x = float_to_bf16_bits(o0) | (float_to_bf16_bits(o1) << 16);
        w.y = float_to_bf16_bits(o2) | (float_to_bf16_bits(o3) << 16);
        *reinterpret_cast<uint2*>(orow + d * 2) = w;
      } else {
        *reinterpret_cast<f32x4*>(orow + d * 4) = f32x4{o0, o1, o2, o3};
      }
    }
  }
  if (hh == 0) a.lse[(int64_t)row * a.n_q_heads + hq] = (m_run * c + __log2f(l)) * kLn2;
}

template <typename T, int D, int GW, bool PREC>
__global__ __launch_bounds__(128 * GW) void attend_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * (Tile<T, D>::kRowBytes +
                                                         (Elem<T>::kBytes == 2 ? Tile<T, D>::kRowBytes
                                                                               : Tile<T, D>::kTBytes))];
  __shared__ int s_sel[64];
  const WgCoord wc = decode_wg(blockIdx.x, a.n_kv_heads, a.gqa / GW);
  // the routing row is requested before anything else
  const RouteRow rrow = load_route_row(a, wc.b, wc.h, threadIdx.x);
  attend_block<T, D, GW, PREC>(a, wc, smem, [&] { return make_routed_set(a, wc.b, rrow, s_sel, threadIdx.x); });
}

// Routing and forward in one launch, for calls whose (query block, kv head)
// pairs alone do not fill the chip: the workgroups of the forward's two-head
// slices each route their block themselves (the routing kernel's single-block
// path, route_blocks with TB = 1), keep the selection in LDS and go on to the
// attention; the first slice writes the routing tables. The query rows the
// routing reads for the block descriptor are the ones the attention reads
// next, and there is one launch fewer per call.
template <typename T, int D, bool PREC>
__global__ __launch_bounds__(256) void route_attend_kernel(RouteArgs ra, AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * (Tile<T, D>::kRowBytes +
                                                         (Elem<T>::kBytes == 2 ? Tile<T, D>::kRowBytes
                                                                               : Tile<T, D>::kTBytes))];
  __shared__ int s_sel[64];
  __shared__ int s_route[65];
  const WgCoord wc = decode_wg(blockIdx.x, a.n_kv_heads, a.gqa / 2);
  attend_block<T, D, 2, PREC>(a, wc, smem, [&] {
    route_blocks<T, D, 1>(ra, wc.b * a.n_kv_heads + wc.h, wc.hs == 0, s_route);
    __syncthreads();  // s_route
    RouteRow row;
    row.nsel = s_route[64];
    row.sel = (int)threadIdx.x < a.top_groups ? s_route[threadIdx.x] : -1;
    return make_routed_set(a, wc.b, row, s_sel, threadIdx.x);
  });
}

template <typename T, int D, bool PREC>
static hipError_t fwd_dispatch(const AttnArgs& a, hipStream_t s) {
  // four query heads per workgroup share each gathered tile; with fewer
  // (block, kv head) pairs than the chip has CUs, two heads per workgroup
  // fill it instead
  int gw = a.gqa >= 4 ? 4 : a.gqa;
  if (gw == 4 && (int64_t)a.n_qb * a.n_kv_heads * (a.gqa / 4) < 256) gw = 2;
  const dim3 grid(a.n_qb * a.n_kv_heads * (a.gqa / gw));
  if (gw == 4)
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 4, PREC>), grid, dim3(512), 0, s, a);
  else if (gw == 2)
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 2, PREC>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 1, PREC>), grid, dim3(128), 0, s, a);
  return hipGetLastError();
}

// The forward's own choice for such calls is two heads per workgroup (see
// fwd_dispatch): G = 2, or G = 4 with fewer than 256 (block, kv head) pairs.
// The fused kernel's static LDS plus the routing's must fit a CU.
bool route_attend_fusable(const AttnArgs& a, size_t route_lds) {
  const bool two_heads = a.gqa == 2 || (a.gqa == 4 && (int64_t)a.n_qb * a.n_kv_heads < 256);
  const size_t fixed = 2 * (2 * Tile<__bf16, 128>::kRowBytes) + 2 * 64 * 4 + 24 * 1024;
  return two_heads && fixed + route_lds <= 160 * 1024;
}

hipError_t launch_route_attend(const RouteArgs& ra, const AttnArgs& a, bool bf16, int head_dim,
                               size_t route_lds, hipStream_t s) {
  const dim3 grid(a.n_qb * a.n_kv_heads * (a.gqa / 2));
#define HGA_RA(T, D, P) hipLaunchKernelGGL((route_attend_kernel<T, D, P>), grid, dim3(256), route_lds, s, ra, a)
  if (bf16) {
    if (head_dim == 64) { if (a.o32) HGA_RA(__bf16, 64, true); else HGA_RA(__bf16, 64, false); }
    else { if (a.o32) HGA_RA(__bf16, 128, true); else HGA_RA(__bf16, 128, false); }
  } else {
    HGA_RA(float, 64, false);  // float32 is built for head_dim 64 only
  }
#undef HGA_RA
  return hipGetLastError();
}

hipError_t launch_attend_fwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s) {
  if (bf16) {
    if (a.o32) return head_dim == 64 ? fwd_dispatch<__bf16, 64, true>(a, s) : fwd_dispatch<__bf16, 128, true>(a, s);
    return head_dim == 64 ? fwd_dispatch<__bf16, 64, false>(a, s) : fwd_dispatch<__bf16, 128, false>(a, s);
  }
  return fwd_dispatch<float, 64, false>(a, s);  // float32 is built for head_dim 64 only
}

}  // namespace hga
