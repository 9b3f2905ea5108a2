// Exact-token routed attention, backward (routing constant: Sec. 2.1 closing
// paragraph; only the active segment gets dK/dV: Sec. 2.2).
//
// With P = softmax(scale * Q K^T) over each query's routed tokens:
//   dP = dO V^T,  D_i = rowsum(dO_i * O_i),  dS = P * (dP - D),
//   dQ = scale * dS K,  dK = scale * dS^T Q,  dV = P^T dO.
//
// One launch runs two kinds of 512-thread workgroups side by side; neither
// waits for the other, so the two run concurrently on the chip, two waves
// per SIMD.
//
// dK/dV role (the first workgroups, dispatched first as they carry the
//     longest chains): key-major, one workgroup per (active 64-token chunk,
//     kv head, subset of query heads). Its eight waves split the work into
//     key half x query half x head-dim half of the accumulators. It holds
//     the chunk's K and V and visits, in
//     ascending order, every query block whose routed set touches the chunk
//     (found by scanning the routing table), for each of the G query heads.
//     D of the visited rows comes from the row-dot kernel run before. The
//     accumulation order is fixed and there are no atomics, so dK/dV are
//     bitwise reproducible, and every active row is written (zero if nothing
//     attends it).
// dQ role: query-major like the forward, one workgroup per (query block, kv
//     head, up to four query heads), gathering the routed K/V tiles into LDS.
#include "routed_tile.h"

namespace hga {

constexpr int kBwdThreads = 512;

template <typename T, int D> struct BwdLds;  // the launch's LDS: the larger of the two roles'

// ---------------------------------------------------------------------------
// dQ role
// ---------------------------------------------------------------------------
template <typename T, int D>
struct DqLayout {
  using TL = Tile<T, D>;
  static constexpr bool TR = Elem<T>::kBytes == 2;  // K^T operand through the LDS transpose load
  static constexpr int STAGE = 2 * TL::kRowBytes + (TR ? 0 : TL::kTBytes);  // K rows, V rows[, K^T]
  static constexpr int OFF_SEL = 2 * STAGE;
  static constexpr int BYTES = OFF_SEL + 64 * 4;
};

// CMP: K and V are the compact routed rows of hga_gather_routed (or the
// tiered gather), [n_qb][Hkv][r_cap][D] in tile order, padding rows zero.
template <typename T, int D, bool CMP = false>
__device__ __forceinline__ void dq_role(const AttnArgs& a, int wg, char* smem) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  using LY = DqLayout<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS, NDT = D / 32, VPS = 16 / E;
  constexpr int NT = kBwdThreads;
  constexpr bool TR = LY::TR;
  constexpr int STAGE = LY::STAGE;
  int* s_sel = reinterpret_cast<int*>(smem + LY::OFF_SEL);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  // up to four query heads per workgroup, two waves (32 queries each) per
  // head; with G < 4 the spare wave pairs repeat a head and write identical
  // rows
  const int gw = a.gqa >= 4 ? 4 : a.gqa;
  const WgCoord wc = decode_wg(wg, a.n_kv_heads, a.gqa / gw);
  const int hq = wc.h * a.gqa + wc.hs * gw + (wave >> 1) % gw;
  const int qoff = (wave & 1) * 32 + l32;
  const int row = wc.b * 64 + qoff;
  // routing row first, then the query-side rows: both in flight together
  const RouteRow rrow = load_route_row(a, wc.b, wc.h, tid);

  Frag qf[NKS], dof[NKS];
  {
    const char* qrow = static_cast<const char*>(a.Q) + ((int64_t)row * a.q_tok + (int64_t)hq * a.q_head) * EB;
    const char* dorow = static_cast<const char*>(a.dO) + ((int64_t)row * a.do_tok + (int64_t)hq * a.do_head) * EB;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int d = ks * KS + E * hh;
      qf[ks] = EL::load_frag(qrow + d * EB);
      dof[ks] = EL::load_frag(dorow + d * EB);
    }
  }
  const float lse2 = a.lse[(int64_t)row * a.n_q_heads + hq] * kLog2e;
  const float Di = a.dvec[(int64_t)row * a.n_q_heads + hq];  // rowsum(dO * O)
  const int64_t cslot = CMP ? ((int64_t)wc.b * a.n_kv_heads + wc.h) * a.r_cap * D * EB : 0;
  const char* kb = static_cast<const char*>(a.K) + (CMP ? cslot : (int64_t)wc.h * a.k_head * EB);
  const char* vb = static_cast<const char*>(a.V) + (CMP ? cslot : (int64_t)wc.h * a.v_head * EB);
  const int64_t ktb = CMP ? D * EB : a.k_tok * EB, vtb = CMP ? D * EB : a.v_tok * EB;
  KVRegs<T, D, NT> kv;
  // the first tile is a window tile: it goes out before the routing row has
  // landed
  RoutedSet rs = window_set(a, wc.b, s_sel);
  kv.load_contiguous(kb, ktb, vb, vtb, CMP ? 0 : rs.window_first(0), tid);
  if (tid < a.top_groups) s_sel[tid] = rrow.sel;
  set_groups(rs, rrow.nsel, s_sel);
  const int ntiles = (rs.R + 63) >> 6;
  __syncthreads();  // s_sel

  f32x16 dqacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) dqacc[dt] = f32x16{};
  const float c = a.scale_log2;
  kv.store_rows(smem, false, tid);
  kv.store_rows(smem + TL::kRowBytes, true, tid);
  if constexpr (!TR) kv.store_transposed(smem + 2 * TL::kRowBytes, false, tid);
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const char* st = smem + (tile & 1) * STAGE;
    if (tile + 1 < ntiles) {
      if constexpr (CMP) kv.load_contiguous(kb, ktb, vb, vtb, (int64_t)64 * (tile + 1), tid);
      else kv.load(kb, ktb, vb, vtb, rs, tile + 1, tid);
    }
    // the same for every lane of the wave; read as a scalar so the masked
    // path is a branch, not a select over every tile
    const bool need_mask = __builtin_amdgcn_readfirstlane((int)rs.tile_needs_mask(tile * 64, (wave & 1) * 32)) != 0;
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
      // masked scores become -inf, whose exponential is exactly 0: a loop of
      // its own under the uniform test, which unmasked tiles branch around
      if (need_mask) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int pos = tile * 64 + 32 * t + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (rs.masked(pos, qoff)) sacc[v] = -__builtin_inff();
        }
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[v], c, -lse2));
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
          if constexpr (TR) kt = tr_frag<TL>(st, 32 * dt, 16 * s + 4 * hh, 16 * s + 8 + 4 * hh, lane);
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

  // dQ rows go through LDS (the stages are free after the loop's last
  // barrier) and leave as 16-byte pieces, consecutive lanes on consecutive
  // pieces of a row; from registers every store would scatter over 32 rows.
  constexpr int OP = D + 4;  // float pitch of a staged row
  static_assert(4 * 64 * OP * 4 <= BwdLds<T, D>::BYTES, "staged dQ rows fit the LDS");
  float* ost = reinterpret_cast<float*>(smem);
  if ((wave >> 1) < gw) {  // spare wave pairs hold copies of these heads
    float* dst = ost + ((wave >> 1) * 64 + qoff) * OP;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4)
        *reinterpret_cast<f32x4*>(dst + 32 * dt + 8 * v4 + 4 * hh) =
            f32x4{dqacc[dt][4 * v4] * a.scale, dqacc[dt][4 * v4 + 1] * a.scale,
                  dqacc[dt][4 * v4 + 2] * a.scale, dqacc[dt][4 * v4 + 3] * a.scale};
  }
  __syncthreads();
  const int hq0 = wc.h * a.gqa + wc.hs * gw;
  constexpr int CPR = D / 4;
  for (int item = tid; item < 64 * gw * CPR; item += NT) {  // (row, head, piece), head fastest after the piece
    const int cc = item % CPR, rj = item / CPR, j = rj % gw, r = rj / gw;
    *reinterpret_cast<f32x4*>(a.dQ + (((int64_t)wc.b * 64 + r) * a.n_q_heads + hq0 + j) * D + 4 * cc) =
        *reinterpret_cast<const f32x4*>(ost + (j * 64 + r) * OP + 4 * cc);
  }
}

// ---------------------------------------------------------------------------
// dK/dV role
// ---------------------------------------------------------------------------

// The head of query block b's routing row for kv head h: its count and first
// sixteen entries, loaded ahead of their use (b < n_qb).
struct MaskRow {
  int nsel;
  int32_t grp[16];
};

__device__ inline MaskRow load_mask_row(const AttnArgs& a, int b, int h) {
  MaskRow r;
  const int64_t slot = (int64_t)b * a.n_kv_heads + h;
  r.nsel = a.n_sel[slot];
  // every load is issued (a branch around them would make the compiler wait
  // for them where the paths join); with no routed groups the first count
  // of the table is read in their place (and the entries are never used)
  const int32_t* sel = a.top_groups > 0 ? a.sel_groups + slot * a.top_groups : a.n_sel;
  const int last = a.top_groups > 0 ? a.top_groups - 1 : 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) r.grp[j] = sel[min(j, last)];
  return r;
}

// Tokens of `chunk` (bit i = token chunk*64 + i) that query block b attends
// through kv head h, from the windows and the routing table (whose head is
// `row`, read ahead).
__device__ inline uint64_t chunk_attend_mask(const AttnArgs& a, int b, int64_t chunk, int h, const MaskRow& row) {
  const int64_t blk_start = a.q_begin + (int64_t)b * 64, blk_end = blk_start + 64;
  const int64_t ls = blk_end - a.local_tokens > 0 ? blk_end - a.local_tokens : 0;
  const int64_t se = a.sink_tokens < ls ? a.sink_tokens : ls;
  const int64_t c0 = chunk * 64;
  if (c0 >= blk_end) return 0;
  if (c0 >= ls) return ~0ull;       // local window (includes the diagonal block)
  if (c0 + 64 <= se) return ~0ull;  // sink window
  const int64_t slot = (int64_t)b * a.n_kv_heads + h;
  const int32_t* sel = a.sel_groups + slot * a.top_groups;
  const int nsel = row.nsel;
  const int g = 1 << a.group_shift;
  const uint64_t gmask = g >= 64 ? ~0ull : ((1ull << g) - 1ull);
  uint64_t m = 0;
  // entries past the first sixteen are read sixteen at a time
  for (int i0 = 0; i0 < a.top_groups; i0 += 16) {
    int32_t grp[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) grp[j] = i0 == 0 ? row.grp[j] : sel[min(i0 + j, a.top_groups - 1)];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int64_t t0 = (int64_t)grp[j] << a.group_shift;
      if (i0 + j < nsel && (t0 >> 6) == chunk) m |= gmask << (t0 & 63);
    }
  }
  return m;
}

// LDS of the key-major role: NST step stages (Q rows, dO rows, [Q^T, dO^T
// for fp32], then lse*log2(e) and D of the 64 query rows), aliased at the end
// by the cross-wave reduction; NXCH P hand-over buffers of the four wave
// pairs; the list of visited query blocks. bf16 reads the transposed operands
// with the LDS transpose load instead of staging them, which leaves room for
// a third stage: the dS/dK wave of a pair then runs one step behind its P/dV
// wave and the two never wait for each other inside a step (PIPE).
template <typename T, int D>
struct StepLayout {
  using TL = Tile<T, D>;
  static constexpr bool TR = Elem<T>::kBytes == 2;
  static constexpr bool PIPE = TR;
  static constexpr int NST = PIPE ? 3 : 2;
  static constexpr int NXCH = PIPE ? 2 : 1;
  static constexpr int OFF_QT = 2 * TL::kRowBytes;
  static constexpr int OFF_OT = OFF_QT + (TR ? 0 : TL::kTBytes);
  static constexpr int OFF_L = OFF_OT + (TR ? 0 : TL::kTBytes);
  static constexpr int OFF_D = OFF_L + 256;
  static constexpr int STAGE = OFF_D + 256;
  static constexpr int RED = 4 * (D / 32) * 16 * 64 * 4;  // cross-wave reduction at the end
  static constexpr int OFF_XCH = NST * STAGE > RED ? NST * STAGE : RED;
  static constexpr int XCH_PAIR = 16 * 64;  // floats per wave pair: P in C layout, [v / 4][lane][4]
  static constexpr int XCH_BUF = 4 * XCH_PAIR;
  static constexpr int OFF_BLK = OFF_XCH + NXCH * XCH_BUF * 4;
  static constexpr int OFF_MASK = OFF_BLK + kBwdThreads * 4;
  static constexpr int OFF_WCOUNT = OFF_MASK + kBwdThreads * 8;
  static constexpr int BYTES = OFF_WCOUNT + 4 * (kBwdThreads / 64);
  static_assert(BYTES <= 160 * 1024, "LDS of the key-major role");
};

// x plus the value of the lane that DPP control CTRL selects (0 where the
// source lane falls outside the row).
template <int CTRL>
__device__ inline float dpp_add(float x) {
  return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

// Sum over each aligned group of N lanes (N = 8 or 16, inside a 16-lane DPP
// row); the total is valid in the group's last lane.
template <int N>
__device__ inline float group_sum_last(float x) {
  static_assert(N == 8 || N == 16, "group of 8 or 16 lanes");
  x = dpp_add<0xB1>(x);                          // quad_perm [1,0,3,2]
  x = dpp_add<0x4E>(x);                          // quad_perm [2,3,0,1]: quad sums
  x = dpp_add<0x114>(x);                         // row_shr:4
  if constexpr (N == 16) x = dpp_add<0x118>(x);  // row_shr:8
  return x;
}

// One thread's share of a step's Q and dO rows (row pairs x 16-byte columns),
// lse and D, prefetched into registers while earlier steps compute.
template <typename T, int D>
struct StepRegs {
  using TL = Tile<T, D>;
  using SL = StepLayout<T, D>;
  static constexpr int EB = Elem<T>::kBytes, E = Elem<T>::E;
  static constexpr int CPR = D * EB / 16;
  static constexpr int NITEMS = 32 * CPR;
  static constexpr int ITEMS = (NITEMS + kBwdThreads - 1) / kBwdThreads;
  u32x4 q[ITEMS][2], o[ITEMS][2];  // native vectors: kept in registers
  // lse and D as loaded: nothing is computed from a prefetched value before
  // the slot is stored (an arithmetic use right after the load would make
  // the compiler wait for it, and for every load issued before it)
  float lse, dd;

  __device__ inline void load(const AttnArgs& a, const int* s_blk, int step, int hq0, int gh, int tid) {
    load_at(a, s_blk[step / gh], hq0 + step % gh, tid);
  }
  __device__ inline void load_at(const AttnArgs& a, int bb, int hq, int tid) {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = min(tid + it * kBwdThreads, NITEMS - 1);  // surplus threads repeat the last item
      const int rp = item / CPR, cc = item % CPR;
      const char* qcol = static_cast<const char*>(a.Q) + (int64_t)hq * a.q_head * EB + cc * 16;
      const char* ocol = static_cast<const char*>(a.dO) + (int64_t)hq * a.do_head * EB + cc * 16;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int64_t r = (int64_t)bb * 64 + 2 * rp + k;
        q[it][k] = *reinterpret_cast<const u32x4*>(row_ptr(qcol, r, a.q_tok * EB));
        o[it][k] = *reinterpret_cast<const u32x4*>(row_ptr(ocol, r, a.do_tok * EB));
      }
    }
    if (tid < 64) {
      const int64_t rh = ((int64_t)bb * 64 + tid) * a.n_q_heads + hq;
      lse = a.lse[rh];
      dd = a.dvec[rh];
    }
  }

  // Rows, lse and D to the stage.
  __device__ inline void store(char* st, int tid) const {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = min(tid + it * kBwdThreads, NITEMS - 1);  // surplus threads rewrite the last item
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
      reinterpret_cast<float*>(st + SL::OFF_L)[tid] = lse * kLog2e;
      reinterpret_cast<float*>(st + SL::OFF_D)[tid] = dd;
    }
  }
};

// The key-major role's step on this wave's 32 queries x 32 keys of the stage
// `st` (query block, query head), shared by the two waves of a (key half,
// query half) pair. Role 0 forms S = Q K^T and P and hands P to its partner
// through LDS, then accumulates dV^T += dO^T P; role 1 forms dP = dO V^T,
// takes P, forms dS = P * (dP - D) and accumulates dK^T += Q^T dS. `kvf`
// holds the wave's K (role 0) or V (role 1) fragments; `acc` covers the whole
// head dim. C layout: lane = key column, rows = queries 32qh + 8(v/4) + 4hh + v%4.

// first product of the step: S (role 0) or dP (role 1), 32 queries x 32 keys
template <typename T, int D>
__device__ __forceinline__ f32x16 dkdv_first(const char* st, const typename Elem<T>::Frag (&kvf)[D / Elem<T>::KSTEP],
                                             int qh, int role, int lane) {
  using EL = Elem<T>;
  using TL = Tile<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, NKS = D / KS;
  const int hh = lane >> 5, l32 = lane & 31;
  f32x16 c = f32x16{};
  const char* arows = st + role * TL::kRowBytes;
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    c = EL::mma(EL::load_frag(arows + TL::row_off(32 * qh + l32, ks * KS + E * hh)), kvf[ks], c);
  return c;
}

// role 0: P from S (masked entries 0) into w and the pair's hand-over buffer
template <typename T, int D>
__device__ __forceinline__ void dkdv_p(const AttnArgs& a, const char* st, float* xch, const f32x16& c,
                                       int64_t blk_start, bool key_on, int64_t ktok, int qh, int lane,
                                       float (&w)[16]) {
  using SL = StepLayout<T, D>;
  const int hh = lane >> 5;
  // the key's position relative to the block's first query, clamped to
  // [-1, 64] (keys before the block are never masked, keys after always)
  const int64_t kd = ktok - blk_start;
  const int kq = kd < -1 ? -1 : kd > 64 ? 64 : (int)kd;
#pragma unroll
  for (int v4 = 0; v4 < 4; ++v4) {
    const f32x4 l4 = *reinterpret_cast<const f32x4*>(st + SL::OFF_L + (32 * qh + 8 * v4 + 4 * hh) * 4);
#pragma unroll
    for (int u = 0; u < 4; ++u) w[4 * v4 + u] = fmaf(c[4 * v4 + u], a.scale_log2, -l4[u]);
  }
  // Hidden entries become -inf (exponential exactly 0). When every key of
  // the wave is attended and precedes all 32 of its queries, which is most
  // steps, the wave branches around the test.
  const bool all_on = __builtin_amdgcn_readfirstlane(__all(key_on && kq <= 32 * qh)) != 0;
  if (!all_on) {
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (!(key_on && kq <= 32 * qh + 8 * (v >> 2) + 4 * hh + (v & 3))) w[v] = -__builtin_inff();
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) w[v] = __builtin_amdgcn_exp2f(w[v]);
  // hand-over layout [v / 4][lane][4]: four 16-byte stores per lane
#pragma unroll
  for (int v4 = 0; v4 < 4; ++v4)
    *reinterpret_cast<f32x4*>(xch + (v4 * 64 + lane) * 4) = f32x4{w[4 * v4], w[4 * v4 + 1], w[4 * v4 + 2], w[4 * v4 + 3]};
}

// role 1: dS = P * (dP - D) from dP and the partner's P
template <typename T, int D>
__device__ __forceinline__ void dkdv_ds(const char* st, const float* xch, const f32x16& c, int qh, int lane,
                                        float (&w)[16]) {
  using SL = StepLayout<T, D>;
  const int hh = lane >> 5;
#pragma unroll
  for (int v4 = 0; v4 < 4; ++v4) {
    const int qr0 = 32 * qh + 8 * v4 + 4 * hh;
    const f32x4 d4 = *reinterpret_cast<const f32x4*>(st + SL::OFF_D + qr0 * 4);
    const f32x4 p4 = *reinterpret_cast<const f32x4*>(xch + (v4 * 64 + lane) * 4);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int v = 4 * v4 + u;
      w[v] = p4[u] * (c[v] - d4[u]);
    }
  }
}

// second product: dV^T += dO^T P (role 0) or dK^T += Q^T dS (role 1)
template <typename T, int D>
__device__ __forceinline__ void dkdv_acc(const char* st, const float (&w)[16], int qh, int role, int lane,
                                         f32x16 (&acc)[D / 32]) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  using SL = StepLayout<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, NDT = D / 32, NQS = 32 / KS;
  const int hh = lane >> 5, l32 = lane & 31;
  const char* trows = st + (role == 0 ? TL::kRowBytes : 0);
  const int off_t = role == 0 ? SL::OFF_OT : SL::OFF_QT;
#pragma unroll
  for (int s = 0; s < NQS; ++s) {
    const Frag f = EL::frag_from(w + E * s);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      Frag t;
      if constexpr (SL::TR) {
        const int ra = 32 * qh + 16 * s + 4 * hh;
        t = tr_frag<TL>(trows, 32 * dt, ra, ra + 8, lane);
      } else {
        t = EL::load_frag(st + off_t + TL::t_off(32 * dt + l32, 32 * qh + KS * s + E * hh));
      }
      acc[dt] = EL::mma(t, f, acc[dt]);
    }
  }
}

template <typename T, int D>
__device__ __forceinline__ void dkdv_role(const AttnArgs& a, int wg, char* smem) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using SL = StepLayout<T, D>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS, NDT = D / 32;
  constexpr int NT = kBwdThreads, NW = NT / 64;
  constexpr int STAGE = SL::STAGE;
  int* s_blk = reinterpret_cast<int*>(smem + SL::OFF_BLK);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(smem + SL::OFF_MASK);
  int* s_wcount = reinterpret_cast<int*>(smem + SL::OFF_WCOUNT);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5, l32 = lane & 31;
  // wave pair (key half, query half); role 0 = P and dV, role 1 = dS and dK
  const int pair = wave & 3, kh = pair & 1, qh = pair >> 1, role = wave >> 2;
  float* xch = reinterpret_cast<float*>(smem + SL::OFF_XCH) + pair * SL::XCH_PAIR;  // + buffer * XCH_BUF
  // work item: (part, chunk, kv head), kv head fastest; part p visits query
  // heads [p * gh, (p + 1) * gh) of the kv head
  const int h = wg % a.n_kv_heads;
  const int cw = (wg / a.n_kv_heads) % a.n_act_chunks;
  const int part = wg / (a.n_kv_heads * a.n_act_chunks);
  const int64_t chunk = a.grad_begin / 64 + cw;
  const int64_t ktok = chunk * 64 + 32 * kh + l32;  // this lane's key token
  const int gh = a.gqa / a.kv_parts;               // query heads visited per block
  const int hq0 = h * a.gqa + part * gh;

  // Everything the first step needs is requested at once: when the chunk's
  // own query block is in the call it is the first block of the list (its
  // local window holds the chunk), so that step's rows go out before the
  // list is built, together with the wave's K or V fragments.
  StepRegs<T, D> sr0, sr1;
  const int b_first = (int)(chunk - a.q_begin / 64 > 0 ? chunk - a.q_begin / 64 : 0);
  const bool early = chunk >= a.q_begin / 64;
  // The routing-table reads of the first list window go out first, then the
  // first step's rows and the K/V fragments: the list waits for the table
  // alone, with the rows still in flight.
  const MaskRow row_first = load_mask_row(a, min(b_first + tid, a.n_qb - 1), h);
  asm volatile("" ::: "memory");  // the table reads are issued before the loads below
  if (early) {
    sr0.load_at(a, b_first, hq0, tid);
  }
  Frag kvf[NKS];
  {
    const int64_t kr = ktok - a.act_begin;  // row of the active-token view
    const char* row = role == 0
        ? static_cast<const char*>(a.Kact) + (kr * a.ka_tok + (int64_t)h * a.ka_head) * EB
        : static_cast<const char*>(a.Vact) + (kr * a.va_tok + (int64_t)h * a.va_head) * EB;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) kvf[ks] = EL::load_frag(row + (ks * KS + E * hh) * EB);
  }
  f32x16 acc[NDT];
#pragma unroll
  for (int j = 0; j < NDT; ++j) acc[j] = f32x16{};
  // the first list window's masks, from the table head read first
  const uint64_t m_first = b_first + tid < a.n_qb ? chunk_attend_mask(a, b_first + tid, chunk, h, row_first) : 0ull;

  // one step = (listed query block, query head): its Q and dO rows, lse, and
  // O for D. Two register slots rotate (two steps' rows in flight while one
  // computes); O is fetched one step ahead of its use.
  for (int base = b_first; base < a.n_qb; base += NT) {
    // ---- list the query blocks of [base, base + NT) that attend this chunk
    const int b = base + tid;
    const uint64_t m = base == b_first ? m_first
        : b < a.n_qb ? chunk_attend_mask(a, b, chunk, h, load_mask_row(a, b, h)) : 0ull;
    const uint64_t ballot = __ballot(m != 0ull);
    const int before = __popcll(ballot & ((1ull << lane) - 1ull));
    __syncthreads();  // the previous list and stages are no longer read
    if (lane == 0) s_wcount[wave] = __popcll(ballot);
    __syncthreads();
    int wbase = 0, n_list = 0;
    for (int w = 0; w < NW; ++w) {
      wbase += w < wave ? s_wcount[w] : 0;
      n_list += s_wcount[w];
    }
    if (m != 0ull) {
      s_blk[wbase + before] = b;
      s_mask[wbase + before] = m;
    }
    const int n_steps = n_list * gh;
    __syncthreads();
    if (n_steps == 0) continue;

    if (!(early && base == b_first)) sr0.load(a, s_blk, 0, hq0, gh, tid);  // else already requested
    // Slot refills are unconditional, on step indices clamped to the last
    // step (a repeated step is loaded and never stored): conditional ones
    // made the compiler wait for both slots before storing either.
    sr1.load(a, s_blk, min(1, n_steps - 1), hq0, gh, tid);
    // step 1's loads stay ahead of step 2's: the loop's stores wait for one
    // slot's loads only when the older slot is always the one stored first
    asm volatile("" ::: "memory");
    sr0.store(smem, tid);
    sr0.load(a, s_blk, min(2, n_steps - 1), hq0, gh, tid);
    __syncthreads();
    // Iteration i: role 0 runs step i; role 1 runs step i - 1 with PIPE (its
    // P was handed over in iteration i - 1), else step i after a barrier.
    // Then the slot holding step i + 1 goes to its stage and the slots refill.
    // Unrolled by two so that every register slot is named statically.
    const int n_iter = n_steps + (SL::PIPE ? 1 : 0);
#define HGA_DKDV_ITER(IT, NEXT)                                                                      \
  {                                                                                                 \
    const int it_ = (IT);                                                                           \
    const int sj_ = SL::PIPE && role == 1 ? it_ - 1 : it_; /* this wave's step */                  \
    const int e_ = sj_ / gh;                                                                        \
    const int64_t bs_ = sj_ >= 0 && sj_ < n_steps ? a.q_begin + (int64_t)s_blk[e_] * 64 : 0;         \
    /* the pair's 32 keys x 32 queries hold a visible entry (with PIPE an */                        \
    /* empty one is skipped by both waves: P and dS are 0 there) */                                 \
    const bool live_ = sj_ >= 0 && sj_ < n_steps &&                                                 \
        (!SL::PIPE || ((uint32_t)(s_mask[e_] >> (32 * kh)) != 0u &&                                 \
                       chunk * 64 + 32 * kh <= bs_ + 32 * qh + 31));                                \
    if (live_) {                                                                                    \
      const char* st = smem + (sj_ % SL::NST) * STAGE;                                              \
      float* xb = xch + (sj_ % SL::NXCH) * SL::XCH_BUF;                                             \
      const f32x16 c = dkdv_first<T, D>(st, kvf, qh, role, lane);                                   \
      float w[16];                                                                                  \
      if (role == 0)                                                                                \
        dkdv_p<T, D>(a, st, xb, c, bs_, (s_mask[e_] >> (32 * kh + l32)) & 1ull, ktok, qh, lane, w); \
      if constexpr (!SL::PIPE) __syncthreads(); /* P of every pair is in LDS */                     \
      if (role == 1) dkdv_ds<T, D>(st, xb, c, qh, lane, w);                                         \
      dkdv_acc<T, D>(st, w, qh, role, lane, acc);                                                   \
    }                                                                                               \
    if (it_ + 1 < n_steps) NEXT.store(smem + ((it_ + 1) % SL::NST) * STAGE, tid); /* step it+1 */    \
    NEXT.load(a, s_blk, min(it_ + 3, n_steps - 1), hq0, gh, tid);         /* refill: step it+3 */    \
    __syncthreads();                                                                                \
  }
    // Whole pairs in the loop and an odd last iteration after it: a loop
    // that could end between the two slots' refills would make the compiler
    // wait for both slots' loads at every store.
    int i0 = 0;
    for (; i0 + 1 < n_iter; i0 += 2) {
      HGA_DKDV_ITER(i0, sr1)
      HGA_DKDV_ITER(i0 + 1, sr0)
    }
    if (i0 < n_iter) HGA_DKDV_ITER(i0, sr1)
#undef HGA_DKDV_ITER
  }

  // ---- sum the two query halves, then write this chunk's rows: role 0
  // holds dV^T, role 1 dK^T, of its key half over the whole head dim
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
  const int slot = kh * 2 + role;
  if (qh == 1) {
#pragma unroll
    for (int j = 0; j < NDT; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) red[((slot * NDT + j) * 16 + v) * 64 + lane] = acc[j][v];
  }
  __syncthreads();
  // The summed rows are staged in LDS as [role][key][D] and leave as 16-byte
  // pieces, consecutive lanes on consecutive pieces of a row (from
  // registers every store would scatter over 32 rows).
  constexpr int OP = D + 4;  // float pitch of a staged row
  static_assert(SL::RED + 2 * 64 * OP * 4 <= SL::BYTES, "staged dK/dV rows fit the LDS");
  float* ost = reinterpret_cast<float*>(smem + SL::RED);
  if (qh == 0) {
    const float mul = role == 0 ? 1.0f : a.scale;
    float* dst = ost + (role * 64 + 32 * kh + l32) * OP;
#pragma unroll
    for (int j = 0; j < NDT; ++j)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        f32x4 r;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int v = 4 * v4 + u;
          r[u] = (acc[j][v] + red[((slot * NDT + j) * 16 + v) * 64 + lane]) * mul;
        }
        *reinterpret_cast<f32x4*>(dst + 32 * j + 8 * v4 + 4 * hh) = r;
      }
  }
  __syncthreads();
  // one work item per (chunk, kv head): the result rows; several: this
  // part's partial rows, summed in part order by the combine kernel
  const int64_t n_rows = (int64_t)a.n_act_chunks * 64 * a.n_kv_heads;
  constexpr int CPR = D / 4;
#pragma unroll
  for (int it = 0; it < 2 * 64 * CPR / NT; ++it) {
    const int item = tid + it * NT;  // (role, key, piece)
    const int cc = item % CPR, k = (item / CPR) % 64, rl = item / (CPR * 64);
    float* out = rl == 0 ? a.dV : a.dK;
    if (a.kv_parts > 1) out = a.part_out + ((int64_t)(rl == 0 ? a.kv_parts : 0) + part) * n_rows * D;
    *reinterpret_cast<f32x4*>(out + ((chunk * 64 + k - a.grad_begin) * a.n_kv_heads + h) * D + 4 * cc) =
        *reinterpret_cast<const f32x4*>(ost + (rl * 64 + k) * OP + 4 * cc);
  }
}

// ---------------------------------------------------------------------------
// The launch: dK/dV workgroups first, then dQ workgroups.
// ---------------------------------------------------------------------------
template <typename T, int D>
struct BwdLds {
  static constexpr int A = StepLayout<T, D>::BYTES, B = DqLayout<T, D>::BYTES;
  static constexpr int BYTES = A > B ? A : B;
};

template <typename T, int D, bool CMP = false>
__global__ __launch_bounds__(kBwdThreads) void bwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[BwdLds<T, D>::BYTES];
  prefetch_args(a);
  const int n_kv = a.kv_parts * a.n_act_chunks * a.n_kv_heads;
  if ((int)blockIdx.x < n_kv) dkdv_role<T, D>(a, blockIdx.x, smem);
  else dq_role<T, D, CMP>(a, blockIdx.x - n_kv, smem);
}

// dK/dV = sum of the kv_parts partials in part order (fixed, so the result
// is reproducible): a streaming pass over both tensors, 16 bytes per thread
// and step.
__global__ __launch_bounds__(256) void bwd_combine_kernel(AttnArgs a, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < 2 * n4; i += stride) {
    const int t = i >= n4;           // 0: dK, 1: dV
    const int64_t j = i - t * n4;    // float4 index inside the tensor
    const f32x4* src = reinterpret_cast<const f32x4*>(a.part_out) + (int64_t)t * a.kv_parts * n4 + j;
    f32x4 acc = src[0];
    for (int p = 1; p < a.kv_parts; ++p) acc += src[(int64_t)p * n4];
    reinterpret_cast<f32x4*>(t == 0 ? a.dK : a.dV)[j] = acc;
  }
}

// D_i = rowsum(dO_i * O_i) of every (query row, query head) into a.dvec
// [n_q][Hq], float32, with O from its float32 copy when there is one. A
// group of TPR consecutive lanes holds one row: 16 bytes of dO per lane.
template <typename T, int D>
__global__ __launch_bounds__(256) void bwd_rowdot_kernel(AttnArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int EPT = 16 / EB;   // elements per lane
  constexpr int TPR = D / EPT;   // lanes per row: 8 or 16
  const int64_t n_pairs = (int64_t)a.n_qb * 64 * a.n_q_heads;
  const int64_t pair = ((int64_t)blockIdx.x * 256 + threadIdx.x) / TPR;
  const int part = threadIdx.x % TPR;
  const int64_t pc = pair < n_pairs ? pair : n_pairs - 1;  // surplus lanes repeat the last row
  const int64_t r = pc / a.n_q_heads;
  const int hq = (int)(pc % a.n_q_heads);
  const u32x4 g = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.dO) +
                                                 (r * a.do_tok + (int64_t)hq * a.do_head) * EB + part * 16);
  float acc = 0.0f;
  if constexpr (EB == 2) {
    float ov[8];
    if (a.o32) {
      const float* src = a.o32 + pc * D + part * 8;
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(src), x1 = *reinterpret_cast<const f32x4*>(src + 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) { ov[j] = x0[j]; ov[4 + j] = x1[j]; }
    } else {
      const u32x4 o = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.O) +
                                                     (r * a.o_tok + (int64_t)hq * a.o_head) * EB + part * 16);
#pragma unroll
      for (int j = 0; j < 8; ++j) ov[j] = bf16_bits_to_float((o[j >> 1] >> ((j & 1) * 16)) & 0xffffu);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = fmaf(bf16_bits_to_float((g[j >> 1] >> ((j & 1) * 16)) & 0xffffu), ov[j], acc);
  } else {
    const f32x4 o = *reinterpret_cast<const f32x4*>(static_cast<const char*>(a.O) +
                                                   (r * a.o_tok + (int64_t)hq * a.o_head) * EB + part * 16);
#pragma unroll
    for (int j = 0; j < 4; ++j) acc = fmaf(__uint_as_float(g[j]), o[j], acc);
  }
  acc = group_sum_last<TPR>(acc);
  if (pair < n_pairs && part == TPR - 1) a.dvec[pair] = acc;
}

template <typename T, int D, bool CMP = false>
static hipError_t bwd_dispatch(const AttnArgs& a, hipStream_t s) {
  {
    constexpr int TPR = D / (16 / Elem<T>::kBytes);
    const int64_t n_pairs = (int64_t)a.n_qb * 64 * a.n_q_heads;
    hipLaunchKernelGGL((bwd_rowdot_kernel<T, D>), dim3((unsigned)((n_pairs * TPR + 255) / 256)), dim3(256), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int gw = a.gqa >= 4 ? 4 : a.gqa;
  const int n_kv = a.kv_parts * a.n_act_chunks * a.n_kv_heads;
  const int n_dq = a.n_qb * a.n_kv_heads * (a.gqa / gw);
  hipLaunchKernelGGL((bwd_kernel<T, D, CMP>), dim3(n_kv + n_dq), dim3(kBwdThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.kv_parts == 1) return e;
  const int64_t n4 = (int64_t)a.n_act_chunks * 64 * a.n_kv_heads * D / 4;  // float4 per tensor
  const int64_t blocks = (2 * n4 + 255) / 256;
  hipLaunchKernelGGL(bwd_combine_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, s, a, n4);
  return hipGetLastError();
}

hipError_t launch_attend_bwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s) {
  if (bf16) return head_dim == 64 ? bwd_dispatch<__bf16, 64>(a, s) : bwd_dispatch<__bf16, 128>(a, s);
  return bwd_dispatch<float, 64>(a, s);  // float32 is built for head_dim 64 only
}

hipError_t launch_attend_gathered_bwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s) {
  if (bf16)
    return head_dim == 64 ? bwd_dispatch<__bf16, 64, true>(a, s) : bwd_dispatch<__bf16, 128, true>(a, s);
  return bwd_dispatch<float, 64, true>(a, s);
}

}  // namespace hga
