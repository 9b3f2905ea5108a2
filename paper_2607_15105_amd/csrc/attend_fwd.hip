// Exact-token routed attention, forward (Sec. 2.1 item 3).
//
// One workgroup per (query block, kv head, slice of GW query heads). Each of
// its 2*GW waves owns 32 queries of one query head. The routed key set
// [sink | local | selected groups] is gathered 64 tokens at a time into LDS,
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
// wc.hs * GW ...), on 2 * GW waves whose thread ids are `tid` (0 .. 128 GW).
// Window tiles (sink and local, known without the routing) come first and
// their gathers go out with the query rows. The selected groups follow:
//  - LATE == false: `routed(rs)` completes rs from the routing row once the
//    window gathers are out; `sync` then makes its LDS writes visible. Three
//    register slots rotate, so tiles t+1..t+3 are in flight while tile t is
//    computed.
//  - LATE == true: the routing is computed by other waves of the workgroup
//    while these attend the window tiles. `ready()` polls whether it has
//    landed (each wave on its own); the gathers of selected groups go out as
//    soon as a wave sees it, and a wave waits for it only when it has no
//    window tile left to compute. Two register slots (the routing waves
//    share the SIMDs' registers).
// Every slot is named statically at each gather and each use (the loop is
// unrolled over the slot rotation), so the compiler waits for exactly the
// gather a use needs and the later ones stay in flight.
// PREC (bf16 only, chosen when the caller asks for the float32 copy of O):
// P enters P.V as a bf16 hi + lo pair, so that copy is accurate to ~2^-17
// relative and the backward's row term D = rowsum(dO * O) is exact enough.
template <typename T, int D, int GW, bool PREC, bool LATE, bool CMP, typename Sync, typename Ready, typename Routed>
__device__ __forceinline__ void attend_block(const AttnArgs& a, const WgCoord wc, char* smem, const int* sel_lds,
                                             const int tid, Sync& sync, Ready&& ready, Routed&& routed) {
  using EL = Elem<T>;
  using Frag = typename EL::Frag;
  using TL = Tile<T, D>;
  // padding keys are masked to -inf below, so their rows need no zeroing
  using KV = KVRegs<T, D, 128 * GW, false>;
  constexpr int E = EL::E, KS = EL::KSTEP, EB = EL::kBytes;
  constexpr int NKS = D / KS;   // MFMAs over the head dim per S tile
  constexpr int NDT = D / 32;   // 32-wide head-dim tiles of O^T
  constexpr int VPS = 16 / E;  // P.V k-steps per 32-key half tile
  constexpr bool TR = EB == 2;  // V operand through the LDS transpose load
  constexpr int STAGE = TL::kRowBytes + (TR ? TL::kRowBytes : TL::kTBytes);

  const int lane = tid & 63, wave = tid >> 6;
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
  // CMP: K and V are the compact copies of hga_gather_routed, rows of this
  // (block, kv head)'s routed set in tile order, padding rows zero
  const int64_t cslot = CMP ? ((int64_t)wc.b * a.n_kv_heads + wc.h) * a.r_cap * D * EB : 0;
  const char* kb = CMP ? Kb + cslot : Kb + k_head_b;
  const char* vb = CMP ? Vb + cslot : Vb + v_head_b;
  const int64_t ktb = CMP ? D * EB : a.k_tok * EB, vtb = CMP ? D * EB : a.v_tok * EB;

  // The query fragments are waited for here, before the tile loop: a first
  // use inside the loop would leave their wait in every iteration, where it
  // also waits for every gather issued after them.
  auto settle = [](Frag (&f)[NKS]) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) asm volatile("" : "+v"(f[ks]));
  };
  RoutedSet rs = window_set(a, wc.b, sel_lds);
  const int nwt = rs.nw >> 6;  // window tiles (>= 1: the diagonal block)
  int ntl = nwt;               // tiles known so far
  bool have = false;           // routing known to this wave
  // gather of tile x into slot r: a window tile before the routing is
  // known, any tile after (rs.token covers both)
  auto gather_w = [&](KV& r, int x) {
    r.load_contiguous(kb, ktb, vb, vtb, CMP ? (int64_t)64 * x : rs.window_first(x), tid);
  };
  auto gather = [&](KV& r, int x) {
    if constexpr (CMP) r.load_contiguous(kb, ktb, vb, vtb, (int64_t)64 * x, tid);
    else if (64 * x < rs.nw) r.load_contiguous(kb, ktb, vb, vtb, rs.window_first(x), tid);
    else r.load_groups(kb, ktb, vb, vtb, rs, x, tid);
  };
  auto take_routing = [&] {
    routed(rs);
    have = true;
    ntl = (rs.R + 63) >> 6;
  };
  auto put = [&](const KV& r, char* dst) {
    r.store_rows(dst, false, tid);
    if constexpr (TR) r.store_rows(dst + TL::kRowBytes, true, tid);
    else r.store_transposed(dst + TL::kRowBytes, true, tid);
  };

  f32x16 oacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) oacc[dt] = f32x16{};
  float m_run = -__builtin_inff(), l_run = 0.0f;
  const float c = a.scale_log2;
  const float lazy = 8.0f / c;  // raise the max only when it grows by > 2^8 in exp2 units

  // One 64-key tile from LDS stage `st` into the running softmax and O, as
  // two 32-key halves, each an online-softmax step of its own: the second
  // half's S products and the first half's P.V products overlap the other
  // half's max and exponentials.
  auto compute = [&](int tile) {
    const char* st = smem + (tile & 1) * STAGE;
    // S^T = K . Q^T : two 32-key tiles, raw scores
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const Frag kf = EL::load_frag(st + TL::row_off(32 * t + l32, ks * KS + E * hh));
        sacc[t] = EL::mma(kf, qf[ks], sacc[t]);
      }
    }
    // the same for every lane of the wave; read as a scalar so the masked
    // path is a branch, not a select over every tile
    const bool need_mask = __builtin_amdgcn_readfirstlane((int)rs.tile_needs_mask(tile * 64, (wave & 1) * 32)) != 0;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (need_mask) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int p = tile * 64 + 32 * t + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (rs.masked(p, qoff)) sacc[t][v] = -__builtin_inff();
        }
      }
      float mx = -__builtin_inff();
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[t][v]);
      mx = fmaxf(mx, xor32(mx));
      const bool raise = mx > m_run + lazy;  // also true on the first half-tile (m_run = -inf)
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
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[t][v], c, -mc));
        sacc[t][v] = p;
        psum += p;
      }
      l_run += psum;
      // O^T += V^T . P^T over this half's keys
#pragma unroll
      for (int s2 = 0; s2 < VPS; ++s2) {
        const int s = t * VPS + s2;
        float pv[E], plo[E];
#pragma unroll
        for (int j = 0; j < E; ++j) {
          pv[j] = sacc[t][E * s2 + j];
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
    }
  };

  if constexpr (!LATE) {
    KV kv0, kv1, kv2;
    gather_w(kv0, 0);  // always a window tile
    if (nwt > 1) gather_w(kv1, 1);
    if (nwt > 2) gather_w(kv2, 2);
    take_routing();
    sync();  // the routing row's LDS copy
    const int ntiles = ntl;
    if (nwt <= 1 && ntiles > 1) gather(kv1, 1);
    if (nwt <= 2 && ntiles > 2) gather(kv2, 2);
    put(kv0, smem);
    if (ntiles > 3) gather(kv0, 3);
    settle(qf);
    sync();
    for (int tile = 0; tile < ntiles; ++tile) {
      compute(tile);
      // the slot holding tile+1 goes to LDS, then refills with tile+4
      if (tile + 1 < ntiles) {
        char* nx = smem + ((tile + 1) & 1) * STAGE;
        const int j = tile % 3;
        if (j == 0) {
          put(kv1, nx);
          if (tile + 4 < ntiles) gather(kv1, tile + 4);
        } else if (j == 1) {
          put(kv2, nx);
          if (tile + 4 < ntiles) gather(kv2, tile + 4);
        } else {
          put(kv0, nx);
          if (tile + 4 < ntiles) gather(kv0, tile + 4);
        }
      }
      sync();
    }
  } else {
    // Slots A, B: tile x lives in kv0 for even x, kv1 for odd x. nl is the
    // next tile to gather; a selected-group tile whose routing this wave has
    // not seen yet waits in nl.
    KV kv0, kv1;
    gather_w(kv0, 0);
    int nl = 1;
    if (nwt > 1) { gather_w(kv1, 1); nl = 2; }
    // next tile x (nl == x) into slot r, if it is known or the routing has
    // landed meanwhile
    auto try_gather = [&](KV& r, int x) {
      if (nl != x) return;
      if (!have && x >= ntl && ready()) take_routing();
      if (x < ntl) { gather(r, x); ++nl; }
    };
    put(kv0, smem);
    try_gather(kv0, 2);
    settle(qf);
    sync();
    // iteration t: compute tile t; tile t+1 (slot A) to LDS; gathers of
    // t+2 (slot B, free since tile t went to LDS) and t+3 (slot A)
    auto iter = [&](int t, KV& A, KV& B) -> bool {
      compute(t);
      if (t + 1 >= ntl) {
        if (have) return false;
        while (!ready()) __builtin_amdgcn_s_sleep(2);
        take_routing();
        if (t + 1 >= ntl) return false;
      }
      if (nl == t + 1) { gather(A, t + 1); ++nl; }  // a selected-group tile not gathered yet
      put(A, smem + ((t + 1) & 1) * STAGE);
      try_gather(B, t + 2);
      try_gather(A, t + 3);
      sync();
      return true;
    };
    for (int tile = 0;; tile += 2) {
      if (!iter(tile, kv1, kv0)) break;
      if (!iter(tile + 1, kv0, kv1)) break;
    }
  }

  // Epilogue: O = O^T / l, LSE = (m + log2 l) * ln 2. A lane holds half the
  // head dim of one query row, so storing from registers would scatter every
  // store instruction over 32 rows; the rows go through LDS instead (the
  // stages are free now), HR query heads at a time, and leave as 16-byte
  // pieces with consecutive lanes on consecutive pieces of a row.
  if constexpr (LATE) sync();  // the last tile's stage is no longer read
  const float l = l_run + xor32(l_run);
  const float inv = 1.0f / l;
  if (hh == 0) a.lse[(int64_t)row * a.n_q_heads + hq] = (m_run * c + __log2f(l)) * kLn2;
  constexpr int OP = D + 4;  // float pitch of a staged row
  constexpr int HR = (2 * STAGE) / (64 * OP * 4) >= GW ? GW : 2;
  static_assert(HR * 64 * OP * 4 <= 2 * STAGE, "staged output rows fit the stages");
  constexpr int NT = 128 * GW;
  float* ost = reinterpret_cast<float*>(smem);
  const int hq0 = wc.h * a.gqa + wc.hs * GW;
#pragma unroll
  for (int r0 = 0; r0 < GW; r0 += HR) {
    if ((wave >> 1) >= r0 && (wave >> 1) < r0 + HR) {
      float* dst = ost + (((wave >> 1) - r0) * 64 + qoff) * OP;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4)
          *reinterpret_cast<f32x4*>(dst + 32 * dt + 8 * v4 + 4 * hh) =
              f32x4{oacc[dt][4 * v4] * inv, oacc[dt][4 * v4 + 1] * inv, oacc[dt][4 * v4 + 2] * inv,
                    oacc[dt][4 * v4 + 3] * inv};
    }
    sync();
    // item = (row r, head j, piece c), head fastest after the piece: with
    // adjacent query heads a row's HR heads are one contiguous run
    {
      constexpr int EPP = 16 / EB;  // elements per 16-byte piece
      constexpr int CPR = D / EPP;
#pragma unroll
      for (int it = 0; it < 64 * HR * CPR / NT; ++it) {
        const int item = tid + it * NT;
        const int cc = item % CPR, rj = item / CPR, j = rj % HR, r = rj / HR;
        const float* src = ost + (j * 64 + r) * OP + cc * EPP;
        char* dst = static_cast<char*>(a.Out) +
                    (((int64_t)wc.b * 64 + r) * a.out_tok + (int64_t)(hq0 + r0 + j) * a.out_head) * EB + cc * 16;
        if constexpr (EB == 2) {
          const f32x4 x0 = *reinterpret_cast<const f32x4*>(src), x1 = *reinterpret_cast<const f32x4*>(src + 4);
          uint4 w;
          w.x = float_to_bf16_bits(x0[0]) | (float_to_bf16_bits(x0[1]) << 16);
          w.y = float_to_bf16_bits(x0[2]) | (float_to_bf16_bits(x0[3]) << 16);
          w.z = float_to_bf16_bits(x1[0]) | (float_to_bf16_bits(x1[1]) << 16);
          w.w = float_to_bf16_bits(x1[2]) | (float_to_bf16_bits(x1[3]) << 16);
          *reinterpret_cast<uint4*>(dst) = w;
        } else {
          *reinterpret_cast<f32x4*>(dst) = *reinterpret_cast<const f32x4*>(src);
        }
      }
    }
    if (a.o32) {
      constexpr int CPR = D / 4;
#pragma unroll
      for (int it = 0; it < 64 * HR * CPR / NT; ++it) {
        const int item = tid + it * NT;
        const int cc = item % CPR, rj = item / CPR, j = rj % HR, r = rj / HR;
        *reinterpret_cast<f32x4*>(a.o32 + (((int64_t)wc.b * 64 + r) * a.n_q_heads + hq0 + r0 + j) * D + 4 * cc) =
            *reinterpret_cast<const f32x4*>(ost + (j * 64 + r) * OP + 4 * cc);
      }
    }
    if (r0 + HR < GW) sync();  // the next heads' rows overwrite these
  }
}

// CMP: over the compact copies of hga_gather_routed (only the routing counts
// are read; the rows come in tile order).
template <typename T, int D, int GW, bool PREC, bool CMP>
__global__ __launch_bounds__(128 * GW) void attend_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * (Tile<T, D>::kRowBytes +
                                                         (Elem<T>::kBytes == 2 ? Tile<T, D>::kRowBytes
                                                                               : Tile<T, D>::kTBytes))];
  __shared__ int s_sel[64];
  prefetch_args(a);
  WgCoord wc = decode_wg(blockIdx.x, a.n_kv_heads, a.gqa / GW);
  // last blocks first when a block's routed set grows with its position (a
  // sink window covering the context, i.e. dense causal attention): the
  // longest workgroups start first and the tail of the grid is short ones
  if (a.heavy_last) wc.b = a.n_qb - 1 - wc.b;
  const int tid = threadIdx.x;
  // the routing row is requested before anything else
  RouteRow rrow;
  if constexpr (CMP) {
    rrow.nsel = a.n_sel[(int64_t)wc.b * a.n_kv_heads + wc.h];
    rrow.sel = -1;
  } else {
    rrow = load_route_row(a, wc.b, wc.h, tid);
  }
  WgSync sync;
  attend_block<T, D, GW, PREC, false, CMP>(a, wc, smem, s_sel, tid, sync, [] { return true; }, [&](RoutedSet& rs) {
    if (tid < a.top_groups) s_sel[tid] = rrow.sel;
    set_groups(rs, rrow.nsel, s_sel);
  });
}

// Routing and forward in one launch, for calls whose (query block, kv head)
// pairs alone do not fill the chip. Each workgroup of a two-head slice has
// eight waves in two teams that run side by side, each with its own barrier:
// waves 0-3 route the block (the routing kernel's single-block path,
// route_blocks with TB = 1; the first slice also writes the routing tables)
// and leave the selection in LDS; waves 4-7 attend the block's window tiles
// meanwhile and take the selected groups as soon as the routing lands.
template <typename T, int D, bool PREC>
__global__ __launch_bounds__(512) void route_attend_kernel(RouteArgs ra, AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * (Tile<T, D>::kRowBytes +
                                                         (Elem<T>::kBytes == 2 ? Tile<T, D>::kRowBytes
                                                                               : Tile<T, D>::kTBytes))];
  __shared__ int s_route[65];  // selected group ids, then their count
  __shared__ int s_sync[3];    // the two teams' barrier counters, the routing-done flag
  prefetch_args(ra);
  prefetch_args(a);
  const WgCoord wc = decode_wg(blockIdx.x, a.n_kv_heads, a.gqa / 2);
  if (threadIdx.x < 3) s_sync[threadIdx.x] = 0;
  __syncthreads();  // the last workgroup-wide barrier: the teams part here
  if (threadIdx.x < 256) {
    WaveGroupSync sync{&s_sync[0], 4};
    // the first summary row goes out after the query rows have landed: the
    // team's waves share the SIMDs' registers with the attention team's
    route_blocks<T, D, 1, false>(ra, wc.b * a.n_kv_heads + wc.h, wc.hs == 0, s_route, (int)threadIdx.x, sync);
    if (threadIdx.x < 64) publish_flag(&s_sync[2]);  // wave 0 wrote s_route
    return;
  }
  const int tid = (int)threadIdx.x - 256;
  WaveGroupSync sync{&s_sync[1], 4};
  attend_block<T, D, 2, PREC, true, false>(a, wc, smem, s_route, tid, sync, [&] { return flag_set(&s_sync[2]); },
                                    [&](RoutedSet& rs) { set_groups(rs, s_route[64], s_route); });
}

template <typename T, int D, bool PREC, bool CMP = false>
static hipError_t fwd_dispatch(const AttnArgs& a, hipStream_t s) {
  // four query heads per workgroup share each gathered tile; with fewer
  // (block, kv head) pairs than the chip has CUs, two heads per workgroup
  // fill it instead
  int gw = a.gqa >= 4 ? 4 : a.gqa;
  if (gw == 4 && (int64_t)a.n_qb * a.n_kv_heads * (a.gqa / 4) < 256) gw = 2;
  const dim3 grid(a.n_qb * a.n_kv_heads * (a.gqa / gw));
  if (gw == 4)
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 4, PREC, CMP>), grid, dim3(512), 0, s, a);
  else if (gw == 2)
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 2, PREC, CMP>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attend_fwd_kernel<T, D, 1, PREC, CMP>), grid, dim3(128), 0, s, a);
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
#define HGA_RA(T, D, P) hipLaunchKernelGGL((route_attend_kernel<T, D, P>), grid, dim3(512), route_lds, s, ra, a)
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

hipError_t launch_attend_gathered_fwd(const AttnArgs& a, bool bf16, int head_dim, hipStream_t s) {
  if (bf16) {
    if (a.o32)
      return head_dim == 64 ? fwd_dispatch<__bf16, 64, true, true>(a, s) : fwd_dispatch<__bf16, 128, true, true>(a, s);
    return head_dim == 64 ? fwd_dispatch<__bf16, 64, false, true>(a, s) : fwd_dispatch<__bf16, 128, false, true>(a, s);
  }
  return fwd_dispatch<float, 64, false, true>(a, s);  // float32 is built for head_dim 64 only
}

}  // namespace hga
