// Exact-token routed attention, forward (Sec. 2.1 item 3).
//
// One workgroup per (query block, kv head, slice of GW query heads). Each of
// its 2*GW waves owns 32 queries of one query head. The routed key set
// [sink | selected groups | local] is gathered 64 tokens at a time into LDS
// (K row-major, V transposed), double-buffered: the next tile's global loads
// are in flight while the matrix cores work on the current one.
//
// Per tile and wave, on 32x32 MFMA tiles:
//   S^T = K . Q^T      (A = K rows from LDS, B = the wave's Q held in registers)
//   online softmax     (every lane holds scores of a single query, so the
//                       running max / sum are per lane plus one cross-half swap)
//   O^T += V^T . P^T   (A = transposed V from LDS, B = P straight from the
//                       S^T accumulators, rounded to the input precision)
// Scores are scaled by softmax_scale*log2(e) and exponentiated with exp2.
#include "routed_tile.h"

namespace hga {

// PREC (bf16 only, chosen when the caller asks for the float32 copy of O):
// P enters P.V as a bf16 hi + lo pair, so that copy is accurate to ~2^-17
// relative and the backward's row term D = rowsum(dO * O) is exact enough.
template <typename T, int D, int GW, bool PREC>
__global__ __launch_bounds__(128 * GW) void attend_fwd_kernel(AttnArgs a) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS;   // MFMAs over the head dim per S tile
  constexpr int NDT = D / 32;   // 32-wide head-dim tiles of O^T
  constexpr int NPS = 64 / KS;  // MFMA k-steps over a 64-key tile in P.V
  constexpr int VPS = 16 / E;
  constexpr int NT = 128 * GW;
  constexpr int STAGE = TL::kRowBytes + TL::kTBytes;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];
  __shared__ int s_sel[64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const WgCoord wc = decode_wg(blockIdx.x, a.n_kv_heads, a.gqa / GW);
  const int hq = wc.h * a.gqa + wc.hs * GW + (wave >> 1);
  const int qoff = (wave & 1) * 32 + l32;  // query offset inside the block
  const int row = wc.b * 64 + qoff;
  const RoutedSet rs = make_routed_set(a, wc.b, wc.h, s_sel, tid, NT);
  const int ntiles = (rs.R + 63) >> 6;

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
  f32x16 oacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) oacc[dt] = f32x16{};
  float m_run = -__builtin_inff(), l_run = 0.0f;

  TileRegs<T, D, NT> kr, vr;
  __syncthreads();  // s_sel
  kr.load(Kb, a.k_tok * EB, k_head_b, rs, 0, tid);
  vr.load(Vb, a.v_tok * EB, v_head_b, rs, 0, tid);
  kr.store_rows(smem, tid);
  vr.store_transposed(smem + TL::kRowBytes, tid);
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const char* st = smem + (tile & 1) * STAGE;
    if (tile + 1 < ntiles) {
      kr.load(Kb, a.k_tok * EB, k_head_b, rs, tile + 1, tid);
      vr.load(Vb, a.v_tok * EB, v_head_b, rs, tile + 1, tid);
    }
    // S^T = K . Q^T : two 32-key tiles
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const Frag kf = EL::load_frag(st + TL::row_off(32 * t + l32, ks * KS + E * hh));
        sacc[t] = EL::mma(kf, qf[ks], sacc[t]);
      }
    }
    // scale, mask, online softmax
    const bool need_mask = rs.tile_needs_mask(tile * 64, (wave & 1) * 32);
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float s = sacc[t][v] * a.scale_log2;
        if (need_mask) {
          const int p = tile * 64 + 32 * t + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (rs.masked(p, qoff)) s = -__builtin_inff();
        }
        sacc[t][v] = s;
        mx = fmaxf(mx, s);
      }
    }
    mx = fmaxf(mx, xor32(mx));
    const float m_new = fmaxf(m_run, mx);
    const float corr = exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= corr;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) oacc[dt] *= corr;
    float psum = 0.0f;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = exp2f(sacc[t][v] - m_new);
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
        const Frag vf = EL::load_frag(st + TL::kRowBytes + TL::t_off(32 * dt + l32, KS * s + E * hh));
        oacc[dt] = EL::mma(vf, pf, oacc[dt]);
        if constexpr (PREC) oacc[dt] = EL::mma(vf, EL::frag_from(plo), oacc[dt]);
      }
    }
    if (tile + 1 < ntiles) {
      char* nx = smem + ((tile + 1) & 1) * STAGE;
      kr.store_rows(nx, tid);
      vr.store_transposed(nx + TL::kRowBytes, tid);
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
  if (hh == 0) a.lse[(int64_t)row * a.n_q_heads + hq] = (m_run + __log2f(l)) * kLn2;
}

template <typename T, int D, bool PREC>
static hipError_t fwd_dispatch(const AttnArgs& a, hipStream_t s) {
  const int gw = a.gqa >= 4 ? 4 : a.gqa;
  const dim3 grid(a.n_qb * a.n_kv_heads * (a.gqa / gw));
  if (gw == 4)
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 4, PREC>), grid, dim3(512), 0, s, a);
  else if (gw == 2)
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 2, PREC>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 1, PREC>), grid, dim3(128), 0, s, a);
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
