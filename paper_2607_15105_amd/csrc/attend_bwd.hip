// Exact-token routed attention, backward (routing constant: Sec. 2.1 closing
// paragraph; only the active segment gets dK/dV: Sec. 2.2).
//
// With P = softmax(scale * Q K^T) over each query's routed tokens:
//   dP = dO V^T,  D_i = rowsum(dO_i * O_i),  dS = P * (dP - D),
//   dQ = scale * dS K,  dK = scale * dS^T Q,  dV = P^T dO.
//
// bwd_dq_kernel   query-major, the same workgroup shape and LDS gather as the
//                 forward (K and V rows plus a transposed K per tile); it
//                 also writes D_i for the second kernel.
// bwd_dkdv_kernel key-major: one workgroup per (active 64-token chunk, kv
//                 head) holds that chunk's K and V and visits, in ascending
//                 order, every query block whose routed set touches the chunk
//                 (found by scanning the routing table), for each of the G
//                 query heads. Accumulation order is fixed and there are no
//                 atomics, so dK/dV are bitwise reproducible, and every active
//                 row is written (zero if nothing attends it).
#include "routed_tile.h"

namespace hga {

template <typename T, int D, int GW>
__global__ __launch_bounds__(128 * GW) void bwd_dq_kernel(AttnArgs a) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS, NDT = D / 32, VPS = 16 / E;
  constexpr int NT = 128 * GW;
  constexpr bool TR = EB == 2;  // K^T operand through the LDS transpose load
  constexpr int STAGE = 2 * TL::kRowBytes + (TR ? 0 : TL::kTBytes);  // K rows, V rows[, K^T]
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];
  __shared__ int s_sel[64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const WgCoord wc = decode_wg(blockIdx.x, a.n_kv_heads, a.gqa / GW);
  const int hq = wc.h * a.gqa + wc.hs * GW + (wave >> 1);
  const int qoff = (wave & 1) * 32 + l32;
  const int row = wc.b * 64 + qoff;
  const RoutedSet rs = make_routed_set(a, wc.b, wc.h, s_sel, tid, NT);
  const int ntiles = (rs.R + 63) >> 6;

  const char* Kb = static_cast<const char*>(a.K);
  const char* Vb = static_cast<const char*>(a.V);
  const int64_t k_head_b = (int64_t)wc.h * a.k_head * EB, v_head_b = (int64_t)wc.h * a.v_head * EB;

  Frag qf[NKS], dof[NKS];
  float Di;
  {
    const char* qrow = static_cast<const char*>(a.Q) + ((int64_t)row * a.q_tok + (int64_t)hq * a.q_head) * EB;
    const char* dorow = static_cast<const char*>(a.dO) + ((int64_t)row * a.do_tok + (int64_t)hq * a.do_head) * EB;
    const char* orow = static_cast<const char*>(a.O) + ((int64_t)row * a.o_tok + (int64_t)hq * a.o_head) * EB;
    const float* o32 = a.o32 ? a.o32 + ((int64_t)row * a.n_q_heads + hq) * D : nullptr;
    float dsum = 0.0f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int d = ks * KS + E * hh;
      qf[ks] = EL::load_frag(qrow + d * EB);
      dof[ks] = EL::load_frag(dorow + d * EB);
      float ov[E];
      if (o32) {
#pragma unroll
        for (int j = 0; j < E; j += (E >= 4 ? 4 : 1)) {
          if constexpr (E >= 4) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(o32 + d + j);
            ov[j] = v[0]; ov[j + 1] = v[1]; ov[j + 2] = v[2]; ov[j + 3] = v[3];
          } else {
            ov[j] = o32[d + j];
          }
        }
      } else {
        const Frag of = EL::load_frag(orow + d * EB);
        if constexpr (E == 1) ov[0] = (float)of;
        else {
#pragma unroll
          for (int j = 0; j < E; ++j) ov[j] = (float)of[j];
        }
      }
      if constexpr (E == 1) {
        dsum += (float)dof[ks] * ov[0];
      } else {
#pragma unroll
        for (int j = 0; j < E; ++j) dsum += (float)dof[ks][j] * ov[j];
      }
    }
    Di = dsum + xor32(dsum);
  }
  const float lse2 = a.lse[(int64_t)row * a.n_q_heads + hq] * kLog2e;
  if (hh == 0) a.Dvec[(int64_t)row * a.n_q_heads + hq] = Di;

  f32x16 dqacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dqacc[dt] = f32x16{};

  KVRegs<T, D, NT> kv;
  const char* kb = Kb + k_head_b;
  const char* vb = Vb + v_head_b;
  const float c = a.scale_log2;
  __syncthreads();
  kv.load(kb, a.k_tok * EB, vb, a.v_tok * EB, rs, 0, tid);
  kv.store_rows(smem, false, tid);
  kv.store_rows(smem + TL::kRowBytes, true, tid);
  if constexpr (!TR) kv.store_transposed(smem + 2 * TL::kRowBytes, false, tid);
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const char* st = smem + (tile & 1) * STAGE;
    if (tile + 1 < ntiles) kv.load(kb, a.k_tok * EB, vb, a.v_tok * EB, rs, tile + 1, tid);
    const bool need_mask = rs.tile_needs_mask(tile * 64, (wave & 1) * 32);
    // the two 32-key halves one after the other: S^T, dP^T, dS^T, then dQ^T
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      f32x16 sacc = f32x16{}, dpacc = f32x16{};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const Frag kf = EL::load_frag(st + TL::row_off(32 * t + l32, ks * KS + E * hh));
        sacc = EL::mma(kf, qf[ks], sacc);
        const Frag vf = EL::load_frag(st + TL::kRowBytes + TL::row_off(32 * t + l32, ks * KS + E * hh));
        dpacc = EL::mma(vf, dof[ks], dpacc);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float p = __builtin_amdgcn_exp2f(fmaf(sacc[v], c, -lse2));
        if (need_mask) {
          const int pos = tile * 64 + 32 * t + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (rs.masked(pos, qoff)) p = 0.0f;
        }
        sacc[v] = p * (dpacc[v] - Di);  // dS^T
      }
      // dQ^T += K^T . dS^T over this half's k-steps. With bf16 inputs dS is
      // carried as a hi + lo pair of bf16 values (two products sharing the K
      // operand): dQ multiplies dS by raw keys, whose magnitude is not
      // bounded, so a single bf16 rounding of dS (2^-9) is not enough.
#pragma unroll
      for (int s2 = 0; s2 < VPS; ++s2) {
        float dv[E], dlo[E];
#pragma unroll
        for (int j = 0; j < E; ++j) {
          dv[j] = sacc[E * s2 + j];
          if constexpr (EB == 2) dlo[j] = dv[j] - bf16_bits_to_float(float_to_bf16_bits(dv[j]));
        }
        const Frag dsf = EL::frag_from(dv);
        const int s = t * VPS + s2;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          Frag kt;
          if constexpr (TR) kt = tr_frag(st, TL::kRowPitch, 32 * dt, 16 * s + 4 * hh, 16 * s + 8 + 4 * hh, lane);
          else kt = EL::load_frag(st + 2 * TL::kRowBytes + TL::t_off(32 * dt + l32, KS * s + E * hh));
          dqacc[dt] = EL::mma(kt, dsf, dqacc[dt]);
          if constexpr (EB == 2) dqacc[dt] = EL::mma(kt, EL::frag_from(dlo), dqacc[dt]);
        }
      }
    }
    if (tile + 1 < ntiles) {
      char* nx = smem + ((tile + 1) & 1) * STAGE;
      kv.store_rows(nx, false, tid);
      kv.store_rows(nx + TL::kRowBytes, true, tid);
      if constexpr (!TR) kv.store_transposed(nx + 2 * TL::kRowBytes, false, tid);
    }
    __syncthreads();
  }

  float* dq = a.dQ + ((int64_t)row * a.n_q_heads + hq) * D;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d = 32 * dt + 8 * v4 + 4 * hh;
      *reinterpret_cast<f32x4*>(dq + d) =
          f32x4{dqacc[dt][4 * v4] * a.scale, dqacc[dt][4 * v4 + 1] * a.scale,
                dqacc[dt][4 * v4 + 2] * a.scale, dqacc[dt][4 * v4 + 3] * a.scale};
    }
  }
}

// Tokens of `chunk` (bit i = token chunk*64 + i) that query block b attends
// through kv head h, from the windows and the routing table. The selected
// groups are scanned without an early exit so their loads issue together.
__device__ inline uint64_t chunk_attend_mask(const AttnArgs& a, int b, int64_t chunk, int h) {
  const int64_t blk_start = a.q_begin + (int64_t)b * 64, blk_end = blk_start + 64;
  const int64_t ls = blk_end - a.local_tokens > 0 ? blk_end - a.local_tokens : 0;
  const int64_t se = a.sink_tokens < ls ? a.sink_tokens : ls;
  const int64_t c0 = chunk * 64;
  if (c0 >= blk_end) return 0;
  if (c0 >= ls) return ~0ull;       // local window (includes the diagonal block)
  if (c0 + 64 <= se) return ~0ull;  // sink window
  const int64_t slot = (int64_t)b * a.n_kv_heads + h;
  const int nsel = a.n_sel[slot];
  const int32_t* sel = a.sel_groups + slot * a.top_groups;
  const int g = 1 << a.group_shift;
  const uint64_t gmask = g >= 64 ? ~0ull : ((1ull << g) - 1ull);
  uint64_t m = 0;
#pragma unroll 8
  for (int i = 0; i < nsel; ++i) {
    const int64_t t0 = (int64_t)sel[i] << a.group_shift;
    if ((t0 >> 6) == chunk) m |= gmask << (t0 & 63);
  }
  return m;
}

// LDS stage of the key-major kernel: Q rows, dO rows, [Q^T, dO^T for fp32],
// then lse*log2(e) and D of the 64 query rows. bf16 reads the transposed
// operands with the LDS transpose load instead of staging them.
template <typename T, int D>
struct StepLayout {
  using TL = Tile<T, D>;
  static constexpr bool TR = Elem<T>::kBytes == 2;
  static constexpr int OFF_QT = 2 * TL::kRowBytes;
  static constexpr int OFF_OT = OFF_QT + (TR ? 0 : TL::kTBytes);
  static constexpr int OFF_L = OFF_OT + (TR ? 0 : TL::kTBytes);
  static constexpr int OFF_D = OFF_L + 256;
  static constexpr int STAGE = OFF_D + 256;
};

// One thread's share of a step's Q and dO rows (row pairs x 16-byte columns),
// prefetched into registers while the previous step computes.
template <typename T, int D>
struct StepRegs {
  using TL = Tile<T, D>;
  using SL = StepLayout<T, D>;
  static constexpr int EB = Elem<T>::kBytes, E = Elem<T>::E;
  static constexpr int CPR = D * EB / 16;
  static constexpr int NITEMS = 32 * CPR;
  static constexpr int ITEMS = NITEMS / 256;
  static_assert(NITEMS % 256 == 0, "staging items must split evenly over 256 threads");
  u32x4 q[ITEMS][2], o[ITEMS][2];  // native vectors: kept in registers
  float lse2, dv;

  __device__ inline void load(const AttnArgs& a, const int* s_blk, int step, int hq0, int gh, int tid) {
    const int bb = s_blk[step / gh];
    const int hq = hq0 + step % gh;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * 256;
      const int rp = item / CPR, cc = item % CPR;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int64_t r = (int64_t)bb * 64 + 2 * rp + k;
        q[it][k] = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.Q) +
                                                  (r * a.q_tok + (int64_t)hq * a.q_head) * EB + cc * 16);
        o[it][k] = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.dO) +
                                                  (r * a.do_tok + (int64_t)hq * a.do_head) * EB + cc * 16);
      }
    }
    if (tid < 64) {
      const int64_t r = (int64_t)bb * 64 + tid;
      lse2 = a.lse[r * a.n_q_heads + hq] * kLog2e;
      dv = a.Dvec[r * a.n_q_heads + hq];
    }
  }

  __device__ inline void store(char* st, int tid) const {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * 256;
      const int rp = item / CPR, cc = item % CPR;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        *reinterpret_cast<u32x4*>(st + TL::row_off(2 * rp + k, cc * 16 / EB)) = q[it][k];
        *reinterpret_cast<u32x4*>(st + TL::kRowBytes + TL::row_off(2 * rp + k, cc * 16 / EB)) = o[it][k];
      }
      if constexpr (!SL::TR) {
        const int kp0 = kpos_of<E>(2 * rp), kp1 = kpos_of<E>(2 * rp + 1);
        const u32x4 qa = q[it][0], qb = q[it][1], oa = o[it][0], ob = o[it][1];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          *reinterpret_cast<uint32_t*>(st + SL::OFF_QT + TL::t_off(cc * 4 + j, kp0)) = qa[j];
          *reinterpret_cast<uint32_t*>(st + SL::OFF_QT + TL::t_off(cc * 4 + j, kp1)) = qb[j];
          *reinterpret_cast<uint32_t*>(st + SL::OFF_OT + TL::t_off(cc * 4 + j, kp0)) = oa[j];
          *reinterpret_cast<uint32_t*>(st + SL::OFF_OT + TL::t_off(cc * 4 + j, kp1)) = ob[j];
        }
      }
    }
    if (tid < 64) {
      reinterpret_cast<float*>(st + SL::OFF_L)[tid] = lse2;
      reinterpret_cast<float*>(st + SL::OFF_D)[tid] = dv;
    }
  }
};

// One step of the key-major kernel: S = Q K^T and dP = dO V^T for this
// wave's 32 queries x 32 keys, then dV^T += dO^T P and dK^T += Q^T dS.
// `st` is the LDS stage of the step (query block, query head).
template <typename T, int D>
__device__ __forceinline__ void dkdv_step(const AttnArgs& a, const char* st, const char* s_kv,
                                          const typename Elem<T>::Frag (&kf)[D / Elem<T>::KSTEP],
                                          const typename Elem<T>::Frag (&vf)[D / Elem<T>::KSTEP],
                                          int64_t blk_start, bool key_on, int64_t ktok, int kh, int qh,
                                          int lane, f32x16 (&dkacc)[D / 32], f32x16 (&dvacc)[D / 32]) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  using SL = StepLayout<T, D>;
  constexpr bool TR = SL::TR;
  constexpr int E = EL::E, KS = EL::KSTEP;
  constexpr int NKS = D / KS, NDT = D / 32, NQS = 32 / KS;
  constexpr int OFF_QT = SL::OFF_QT, OFF_OT = SL::OFF_OT, OFF_L = SL::OFF_L, OFF_D = SL::OFF_D;
  const int hh = lane >> 5, l32 = lane & 31;
    // ---- S = Q K^T and dP = dO V^T for 32 queries x 32 keys
    f32x16 sacc = f32x16{}, dpacc = f32x16{};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const Frag qa = EL::load_frag(st + TL::row_off(32 * qh + l32, ks * KS + E * hh));
      const Frag oa = EL::load_frag(st + TL::kRowBytes + TL::row_off(32 * qh + l32, ks * KS + E * hh));
      Frag kb, vb;
      if constexpr (TR) {
        kb = EL::load_frag(s_kv + TL::row_off(32 * kh + l32, ks * KS + E * hh));
        vb = EL::load_frag(s_kv + TL::kRowBytes + TL::row_off(32 * kh + l32, ks * KS + E * hh));
      } else {
        kb = kf[ks];
        vb = vf[ks];
      }
      sacc = EL::mma(qa, kb, sacc);
      dpacc = EL::mma(oa, vb, dpacc);
    }
    // lane: key column; rows: queries 32qh + 8(v/4) + 4hh + v%4
    float pv[16], dsv[16];
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int qr0 = 32 * qh + 8 * v4 + 4 * hh;
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(st + OFF_L + qr0 * 4);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(st + OFF_D + qr0 * 4);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = 4 * v4 + u;
        const bool on = key_on && ktok <= blk_start + qr0 + u;
        const float p = on ? __builtin_amdgcn_exp2f(fmaf(sacc[v], a.scale_log2, -l4[u])) : 0.0f;
        pv[v] = p;
        dsv[v] = p * (dpacc[v] - d4[u]);
      }
    }
    // ---- dV^T += dO^T P,  dK^T += Q^T dS
#pragma unroll
    for (int s = 0; s < NQS; ++s) {
      const Frag pf = EL::frag_from(pv + E * s);
      const Frag df = EL::frag_from(dsv + E * s);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        Frag ot, qt;
        if constexpr (TR) {
          const int ra = 32 * qh + 16 * s + 4 * hh;
          ot = tr_frag(st + TL::kRowBytes, TL::kRowPitch, 32 * dt, ra, ra + 8, lane);
          qt = tr_frag(st, TL::kRowPitch, 32 * dt, ra, ra + 8, lane);
        } else {
          const int kp = 32 * qh + KS * s + E * hh;
          ot = EL::load_frag(st + OFF_OT + TL::t_off(32 * dt + l32, kp));
          qt = EL::load_frag(st + OFF_QT + TL::t_off(32 * dt + l32, kp));
        }
        dvacc[dt] = EL::mma(ot, pf, dvacc[dt]);
        dkacc[dt] = EL::mma(qt, df, dkacc[dt]);
      }
    }}

template <typename T, int D>
__global__ __launch_bounds__(256) void bwd_dkdv_kernel(AttnArgs a) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS, NDT = D / 32;
  using SL = StepLayout<T, D>;
  constexpr bool TR = SL::TR;
  constexpr int STAGE = SL::STAGE;
  constexpr int RED = 2 * 64 * NDT * 16 * 2 * 4;  // cross-wave reduction at the end
  constexpr int SMEM = 2 * STAGE > RED ? 2 * STAGE : RED;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  // bf16: the chunk's K and V rows live in LDS (B operands of S and dP);
  // fp32 keeps them in registers, its LDS holds the transposed staging.
  __shared__ __attribute__((aligned(16))) char s_kv[TR ? 2 * TL::kRowBytes : 16];
  __shared__ int s_blk[256];
  __shared__ uint64_t s_mask[256];
  __shared__ int s_wcount[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int kh = wave & 1, qh = wave >> 1;
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t chunk = a.grad_begin / 64 + blockIdx.x / a.n_kv_heads;
  const int64_t ktok = chunk * 64 + 32 * kh + l32;  // this lane's key token
  const int gh = a.gqa;                             // query heads visited per block
  const int hq0 = h * a.gqa;

  // the chunk's K and V as B operands (column = key, k = head dim)
  Frag kf[NKS], vf[NKS];
  if constexpr (TR) {
    constexpr int CPR = D * EB / 16;
    for (int item = tid; item < 2 * 64 * CPR; item += 256) {
      const int m = item / (64 * CPR), r = (item / CPR) % 64, cc = item % CPR;
      const int64_t t = chunk * 64 + r;
      const char* src = m == 0 ? static_cast<const char*>(a.K) + (t * a.k_tok + (int64_t)h * a.k_head) * EB
                               : static_cast<const char*>(a.V) + (t * a.v_tok + (int64_t)h * a.v_head) * EB;
      *reinterpret_cast<uint4*>(s_kv + m * TL::kRowBytes + TL::row_off(r, cc * 16 / EB)) =
          *reinterpret_cast<const uint4*>(src + cc * 16);
    }
  } else {
    const char* krow = static_cast<const char*>(a.K) + (ktok * a.k_tok + (int64_t)h * a.k_head) * EB;
    const char* vrow = static_cast<const char*>(a.V) + (ktok * a.v_tok + (int64_t)h * a.v_head) * EB;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      kf[ks] = EL::load_frag(krow + (ks * KS + E * hh) * EB);
      vf[ks] = EL::load_frag(vrow + (ks * KS + E * hh) * EB);
    }
  }
  f32x16 dkacc[NDT], dvacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dkacc[dt] = dvacc[dt] = f32x16{};

  // one step = (listed query block, query head): its Q and dO rows, lse, D
  // three register slots rotate: three steps' loads in flight while one computes
  StepRegs<T, D> sr0, sr1, sr2;
  const int b_first = (int)(chunk - a.q_begin / 64 > 0 ? chunk - a.q_begin / 64 : 0);
  for (int base = b_first; base < a.n_qb; base += 256) {
    // ---- list the query blocks of [base, base+256) that attend this chunk
    const int b = base + tid;
    const uint64_t m = b < a.n_qb ? chunk_attend_mask(a, b, chunk, h) : 0ull;
    const uint64_t ballot = __ballot(m != 0ull);
    const int before = __popcll(ballot & ((1ull << lane) - 1ull));
    __syncthreads();  // the previous list and stages are no longer read
    if (lane == 0) s_wcount[wave] = __popcll(ballot);
    __syncthreads();
    int wbase = 0;
    for (int w = 0; w < wave; ++w) wbase += s_wcount[w];
    if (m != 0ull) {
      s_blk[wbase + before] = b;
      s_mask[wbase + before] = m;
    }
    const int n_steps = (s_wcount[0] + s_wcount[1] + s_wcount[2] + s_wcount[3]) * gh;
    __syncthreads();
    if (n_steps == 0) continue;

    sr0.load(a, s_blk, 0, hq0, gh, tid);
    if (n_steps > 1) sr1.load(a, s_blk, 1, hq0, gh, tid);
    if (n_steps > 2) sr2.load(a, s_blk, 2, hq0, gh, tid);
    sr0.store(smem, tid);
    if (n_steps > 3) sr0.load(a, s_blk, 3, hq0, gh, tid);
    __syncthreads();
    // unrolled by three so that every register slot is named statically
#define HGA_DKDV_STEP(STEP, NEXT)                                                                    \
  if ((STEP) < n_steps) {                                                                           \
    const int step_ = (STEP);                                                                       \
    const int e_ = step_ / gh;                                                                      \
    dkdv_step<T, D>(a, smem + (step_ & 1) * STAGE, s_kv, kf, vf, a.q_begin + (int64_t)s_blk[e_] * 64, \
                    (s_mask[e_] >> (32 * kh + l32)) & 1ull, ktok, kh, qh, lane, dkacc, dvacc);      \
    if (step_ + 1 < n_steps) { /* slot with step+1 -> LDS, refill with step+4 */                  \
      NEXT.store(smem + ((step_ + 1) & 1) * STAGE, tid);                                            \
      if (step_ + 4 < n_steps) NEXT.load(a, s_blk, step_ + 4, hq0, gh, tid);                        \
    }                                                                                               \
    __syncthreads();                                                                                \
  }
    for (int s0 = 0; s0 < n_steps; s0 += 3) {
      HGA_DKDV_STEP(s0, sr1)
      HGA_DKDV_STEP(s0 + 1, sr2)
      HGA_DKDV_STEP(s0 + 2, sr0)
    }
#undef HGA_DKDV_STEP
  }

  // ---- sum the two query halves, then write this chunk's rows
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
  if (qh == 1) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        red[((kh * 2 + 0) * NDT * 16 + dt * 16 + v) * 64 + lane] = dkacc[dt][v];
        red[((kh * 2 + 1) * NDT * 16 + dt * 16 + v) * 64 + lane] = dvacc[dt][v];
      }
  }
  __syncthreads();
  if (qh == 0) {
    const int64_t orow = ((ktok - a.grad_begin) * a.n_kv_heads + h) * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        f32x4 k4, v4v;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int v = 4 * v4 + u;
          k4[u] = (dkacc[dt][v] + red[((kh * 2 + 0) * NDT * 16 + dt * 16 + v) * 64 + lane]) * a.scale;
          v4v[u] = dvacc[dt][v] + red[((kh * 2 + 1) * NDT * 16 + dt * 16 + v) * 64 + lane];
        }
        const int d = 32 * dt + 8 * v4 + 4 * hh;
        *reinterpret_cast<f32x4*>(a.dK + orow + d) = k4;
        *reinterpret_cast<f32x4*>(a.dV + orow + d) = v4v;
      }
  }
}

template <typename T, int D>
static hipError_t bwd_dispatch(const AttnArgs& a, hipStream_t s) {
  const int gw = a.gqa >= 4 ? 4 : a.gqa;
  const dim3 grid(a.n_qb * a.n_kv_heads * (a.gqa / gw));
  if (gw == 4)
    hipLaunchKernelGGL((bwd_dq_kernel<T, D, 4>), grid, dim3(512), 0, s, a);
  else if (gw == 2)
    hipLaunchKernelGGL((bwd_dq_kernel<T, D, 2>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_dq_kernel<T, D, 1>), grid, dim3(128), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((bwd_dkdv_kernel<T, D>), dim3(a.n_act_chunks * a.n_kv_heads), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attend_bwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s) {
  if (bf16) return head_dim == 64 ? bwd_dispatch<__bf16, 64>(a, s) : bwd_dispatch<__bf16, 128>(a, s);
  return bwd_dispatch<float, 64>(a, s);  // float32 is built for head_dim 64 only
}

}  // namespace hga
