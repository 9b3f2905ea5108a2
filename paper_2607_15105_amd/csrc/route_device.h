// Two-level routing (Sec. 2.1 items 1-2, Fig. 1), device code shared by the
// routing kernel and the fused routing + forward kernel. A workgroup of four
// waves handles TB consecutive query blocks of one kv head:
//
//   phase 0  block descriptor qbar = mean of the block's B rows over the G
//            query heads of the kv head, summed exactly in float64 (bf16 has
//            8 significant bits) and scaled by 1/(B*G), a power of two;
//   phase 1  chunk scores qbar . s^C for every candidate chunk of the TB
//            blocks. Lane = chunk: a lane reads its summary row in units
//            (halves or quarters) that run ahead of the arithmetic, and
//            scores each unit against all TB descriptors (each row is read
//            once per workgroup);
//   phase 2  top-k_c per block, one wave per block (wave_top_k below);
//   phase 3  group scores qbar . s^G over all groups of the chosen chunks;
//   phase 4  global top-k_g per block over those groups.
//
// Scores are float64 FMA chains in head-dim order. Selection order: larger
// score first, lower index on equal scores (NaN scores count as -inf); the
// selected sets are returned ascending.
#pragma once
#include "hga_device.h"
#include "hga_kernels.h"

namespace hga {

constexpr int kNoIdx = 0x7fffffff;
constexpr int kListCap = 256;  // entries a wave ranks directly

__device__ inline bool better(double va, int ia, double vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// Number of set bits of m below this lane.
__device__ inline int lanes_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ inline double readlane_d(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ inline double shfl_xor_d(double v, int m) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const int lo = __shfl_xor((int)(uint32_t)u, m, 64);
  const int hi = __shfl_xor((int)(uint32_t)(u >> 32), m, 64);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

__device__ inline double no_nan(double x) { return x == x ? x : -__builtin_inf(); }

// LDS scratch of one wave's selection.
struct TopKScratch {
  double lbv[64];        // lane bests
  int lbi[64];
  double lv[kListCap];   // entries at or above the threshold, ascending index
  int li[kListCap];
  int out[64];           // selected positions, ascending
};

// Slow exact selection for inputs the threshold cannot narrow to kListCap
// entries: k rounds of a wave-wide arg-best over cached per-lane top-2 lists.
// An entry is still available when it comes strictly after the last winner.
struct Top2 {
  double v1, v2;
  int i1, i2;
};

__device__ inline Top2 lane_top2_after(const double* sc, int n, int lane, double wv, int wi) {
  Top2 t{-__builtin_inf(), -__builtin_inf(), kNoIdx, kNoIdx};
  for (int i = lane; i < n; i += 64) {
    const double v = sc[i];
    if (!better(wv, wi, v, i)) continue;
    if (better(v, i, t.v1, t.i1)) { t.v2 = t.v1; t.i2 = t.i1; t.v1 = v; t.i1 = i; }
    else if (better(v, i, t.v2, t.i2)) { t.v2 = v; t.i2 = i; }
  }
  return t;
}

__device__ __attribute__((always_inline)) inline int top_k_tournament(const double* sc, int n,
                                                                      int k_eff, int lane) {
  double wv = __builtin_inf();
  int wi = -1;
  Top2 t = lane_top2_after(sc, n, lane, wv, wi);
  int mine = kNoIdx;
  for (int r = 0; r < k_eff; ++r) {
    double bv = t.v1;
    int bi = t.i1;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const double ov = shfl_xor_d(bv, m);
      const int oi = __shfl_xor(bi, m, 64);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == r) mine = bi;
    wv = bv;
    wi = bi;
    bool rescan = false;
    if (t.i1 == bi) {  // this lane held the winner
      t.v1 = t.v2; t.i1 = t.i2;
      t.v2 = -__builtin_inf(); t.i2 = kNoIdx;
      rescan = (t.i1 == kNoIdx);
    }
    if (__any(rescan)) {
      const Top2 u = lane_top2_after(sc, n, lane, wv, wi);
      if (rescan) t = u;
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

// Branch-free form of `better` for values already in registers (the
// short-circuit form makes the compiler fetch the index behind a branch).
__device__ inline bool better_nb(double va, int ia, double vb, int ib) {
  return (va > vb) | ((va == vb) & (ia < ib));
}

// Rank of (mv, mi) among the first L entries of (lv, li): the number of
// entries that come before it. Entries are read in batches of 8 so their
// LDS round trips overlap; the arrays hold at least round_up(L, 8) entries.
__device__ inline int rank_among(const double* lv, const int* li, int L, double mv, int mi) {
  int rk = 0;
#pragma unroll 1
  for (int j0 = 0; j0 < L; j0 += 8) {
    double v[8];
    int ix[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) { v[u] = lv[j0 + u]; ix[u] = li[j0 + u]; }
#pragma unroll
    for (int u = 0; u < 8; ++u) rk += ((j0 + u < L) & better_nb(v[u], ix[u], mv, mi)) ? 1 : 0;
  }
  return rk;
}

// Entries lane + 64 e (e < EPL) of the list ranked in one pass over it; the
// ones ranked below k_eff go to ws.out in list (= index) order. Returns how
// many were selected.
template <int EPL>
__device__ inline int rank_select(TopKScratch& ws, int L, int k_eff, int lane) {
  double mv[EPL];
  int mi[EPL], rk[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    mv[e] = ws.lv[lane + 64 * e];
    mi[e] = ws.li[lane + 64 * e];
    rk[e] = 0;
  }
#pragma unroll 1
  for (int j0 = 0; j0 < L; j0 += 8) {
    double v[8];
    int ix[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) { v[u] = ws.lv[j0 + u]; ix[u] = ws.li[j0 + u]; }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < EPL; ++e) rk[e] += ((j0 + u < L) & better_nb(v[u], ix[u], mv[e], mi[e])) ? 1 : 0;
  }
  int nsel = 0;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    const bool sel = (lane + 64 * e < L) & (rk[e] < k_eff);
    const uint64_t ms = __ballot(sel);
    const int pos = nsel + lanes_below(ms);
    if (sel && pos < 64) ws.out[pos] = mi[e];
    nsel += __popcll(ms);
  }
  return nsel;
}

// Top-k (k <= 64) positions of the scores sc[0..n) (no NaN), returned
// ascending: lane r < min(k, n) gets the r-th smallest selected position,
// the other lanes kNoIdx. Called by a whole wave; sc is not modified.
//
// When n > 64 the k-th best of the 64 lane bests (each lane's best over its
// strided slice) is a threshold: the k lane bests at or above it are k
// entries, so every top-k entry is at or above it too. The entries at or
// above the threshold are compacted in index order (at most k lane slices
// contribute, so n <= 256 always fits kListCap) and ranked exactly: an
// entry's rank among them equals its rank among all n.
__device__ __attribute__((always_inline)) inline int wave_top_k(const double* sc, int n, int k,
                                                                int lane, TopKScratch& ws) {
  const int k_eff = min(k, n);
  if (k_eff <= 0) return kNoIdx;
  if (k_eff == n) return lane < n ? lane : kNoIdx;  // take all (n <= 64)
  int L;
  if (n <= 64) {
    ws.lv[lane] = lane < n ? sc[lane] : -__builtin_inf();
    ws.li[lane] = lane < n ? lane : kNoIdx;
    L = n;
  } else {
    double bv = -__builtin_inf();
    int bi = kNoIdx;
    for (int i0 = lane; i0 < n; i0 += 256) {
      double v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = sc[min(i0 + 64 * u, n - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int p = i0 + 64 * u;
        const bool b = (p < n) & better_nb(v[u], p, bv, bi);
        bv = b ? v[u] : bv;
        bi = b ? p : bi;
      }
    }
    ws.lbv[lane] = bv;
    ws.lbi[lane] = bi;
    __builtin_amdgcn_wave_barrier();
    const int rk = rank_among(ws.lbv, ws.lbi, 64, bv, bi);
    const uint64_t mt = __ballot(rk == k_eff - 1);
    const int tl = __builtin_ctzll(mt);
    const double tv = readlane_d(bv, tl);
    const int ti = __builtin_amdgcn_readlane(bi, tl);
    int base = 0;
    for (int j0 = 0; j0 < n; j0 += 256) {
      double v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = sc[min(j0 + 64 * u + lane, n - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int p = j0 + 64 * u + lane;
        const bool q = (p < n) & ((p == ti) | better_nb(v[u], p, tv, ti));
        const uint64_t mq = __ballot(q);
        const int pos = base + lanes_below(mq);
        if (q && pos < kListCap) { ws.lv[pos] = v[u]; ws.li[pos] = p; }
        base += __popcll(mq);
      }
    }
    if (base > kListCap) return top_k_tournament(sc, n, k_eff, lane);
    L = base;
  }
  __builtin_amdgcn_wave_barrier();
  // rank of each list entry; this lane holds entries lane + 64 e
  int nsel = 0;
  if (L <= 64) {
    const double mv = ws.lv[lane];
    const int mi = ws.li[lane];
    const bool sel = (lane < L) & (rank_among(ws.lv, ws.li, L, mv, mi) < k_eff);
    const uint64_t ms = __ballot(sel);
    if (sel) ws.out[lanes_below(ms)] = mi;
    nsel = __popcll(ms);
  } else if (L <= 128) {
    nsel = rank_select<2>(ws, L, k_eff, lane);
  } else {
    nsel = rank_select<kListCap / 64>(ws, L, k_eff, lane);
  }
  __builtin_amdgcn_wave_barrier();
  // nsel == k_eff: ranks of distinct entries under a total order are distinct
  return lane < k_eff && lane < nsel ? ws.out[lane] : kNoIdx;
}

// wave_top_k for a workgroup that routes a single block: all four waves call
// it with the same arguments and share the rank comparisons (each compares
// against a quarter of the entries; wave 0 adds the four partial ranks);
// wave 0 does the rest. The result lands in wave 0's lanes as wave_top_k's
// does; the other waves get kNoIdx.
template <typename Sync>
__device__ __attribute__((always_inline)) inline int block_top_k(const double* sc, int n, int k, int wave,
                                                                 int lane, TopKScratch& ws, int (*s_part)[64],
                                                                 int* s_len, Sync& sync) {
  const int k_eff = min(k, n);
  if (k_eff <= 0) return kNoIdx;
  if (k_eff == n) return wave == 0 && lane < n ? lane : kNoIdx;  // take all (n <= 64)
  if (n <= 64) {
    if (wave == 0) {
      ws.lv[lane] = lane < n ? sc[lane] : -__builtin_inf();
      ws.li[lane] = lane < n ? lane : kNoIdx;
    }
  } else {
    // threshold: the k-th best of the 64 lane bests (see wave_top_k)
    double bv = -__builtin_inf();
    int bi = kNoIdx;
    if (wave == 0) {
      for (int i0 = lane; i0 < n; i0 += 256) {
        double v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = sc[min(i0 + 64 * u, n - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int p = i0 + 64 * u;
          const bool b = (p < n) & better_nb(v[u], p, bv, bi);
          bv = b ? v[u] : bv;
          bi = b ? p : bi;
        }
      }
      ws.lbv[lane] = bv;
      ws.lbi[lane] = bi;
    }
    sync();
    s_part[wave][lane] = rank_among(ws.lbv + 16 * wave, ws.lbi + 16 * wave, 16, ws.lbv[lane], ws.lbi[lane]);
    sync();
    if (wave == 0) {
      const int rk = s_part[0][lane] + s_part[1][lane] + s_part[2][lane] + s_part[3][lane];
      const uint64_t mt = __ballot(rk == k_eff - 1);
      const int tl = __builtin_ctzll(mt);
      const double tv = readlane_d(bv, tl);
      const int ti = __builtin_amdgcn_readlane(bi, tl);
      int base = 0;
      for (int j0 = 0; j0 < n; j0 += 256) {
        double v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = sc[min(j0 + 64 * u + lane, n - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int p = j0 + 64 * u + lane;
          const bool q = (p < n) & ((p == ti) | better_nb(v[u], p, tv, ti));
          const uint64_t mq = __ballot(q);
          const int pos = base + lanes_below(mq);
          if (q && pos < kListCap) { ws.lv[pos] = v[u]; ws.li[pos] = p; }
          base += __popcll(mq);
        }
      }
      if (lane == 0) *s_len = base;
    }
  }
  sync();  // the list to rank
  const int L = n <= 64 ? n : *s_len;
  if (L > kListCap) return wave == 0 ? top_k_tournament(sc, n, k_eff, lane) : kNoIdx;
  int nsel = 0;
  if (L <= 64) {
    const int lo = 16 * wave, cnt = max(0, min(16, L - lo));
    s_part[wave][lane] = rank_among(ws.lv + lo, ws.li + lo, cnt, ws.lv[lane], ws.li[lane]);
    sync();
    if (wave == 0) {
      const int rk = s_part[0][lane] + s_part[1][lane] + s_part[2][lane] + s_part[3][lane];
      const bool sel = (lane < L) & (rk < k_eff);
      const uint64_t ms = __ballot(sel);
      if (sel) ws.out[lanes_below(ms)] = ws.li[lane];
      nsel = __popcll(ms);
    }
  } else if (wave == 0) {
    nsel = L <= 128 ? rank_select<2>(ws, L, k_eff, lane) : rank_select<kListCap / 64>(ws, L, k_eff, lane);
  }
  if (wave != 0) return kNoIdx;
  __builtin_amdgcn_wave_barrier();
  return lane < k_eff && lane < nsel ? ws.out[lane] : kNoIdx;
}

// One past the last candidate chunk of absolute query block `blk`: chunks end
// at or before the start of the block's local window.
__device__ inline int last_cand(int64_t blk, int local_tokens) {
  const int64_t ls = (blk + 1) * 64 - local_tokens;
  return ls > 0 ? (int)(ls / 64) : 0;
}

// Summary rows are scored one row per lane, in UPR units (quarters or
// halves) of D/(4 UPR) quads: the unit loads of a lane's sequence of (pass,
// unit) run ahead of the arithmetic in two or three register slots. With the
// quad-major tables the lanes of one load instruction read consecutive rows'
// quads (64 contiguous 16-byte pieces).
template <int D, int UPR>
__device__ inline void load_unit(f32x4 (&v)[D / 4 / UPR], const float* table, int64_t r, int64_t cap, int u) {
  constexpr int QPU = D / 4 / UPR;
  const f32x4* t = reinterpret_cast<const f32x4*>(table) + r;
#pragma unroll
  for (int k = 0; k < QPU; ++k) v[k] = t[(int64_t)(u * QPU + k) * cap];
}

// a0/a1[t] += unit u of a row . unit u of descriptor t, for the blocks
// t < nb: two float64 FMA chains per block over the head dim. The row is
// converted to double 16 values at a time, once for all blocks.
template <int D, int UPR, int TB>
__device__ inline void unit_dots(f32x4 (&v)[D / 4 / UPR], const double (*desc)[D], int u, int nb,
                                 double (&a0)[TB], double (&a1)[TB]) {
  constexpr int QPU = D / 4 / UPR;
#pragma unroll
  for (int g = 0; g < QPU / 4; ++g) {
    // the conversions of a group are not moved ahead of it (nor out of the
    // caller's loop): they never hold more than 16 doubles
#pragma unroll
    for (int w = 0; w < 4; ++w) asm volatile("" : "+v"(v[4 * g + w]));
    double x[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) x[e] = (double)v[4 * g + e / 4][e % 4];
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      if (t < nb) {
        const double* qp = desc[t] + u * (D / UPR) + 16 * g;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
          const double2 qd = *reinterpret_cast<const double2*>(qp + e);
          a0[t] = fma(x[e], qd.x, a0[t]);
          a1[t] = fma(x[e + 1], qd.y, a1[t]);
        }
      }
    }
  }
}

// Routing of the TB query blocks of workgroup `wg` on four waves whose thread
// ids are `tid` (0..255) and whose barrier is `sync`, in the phases
// described at the top. EARLY_ROW (TB == 1 only): the first chunk-summary
// rows are requested before the query rows (else once the query rows have
// been summed, which keeps their registers free while the query rows are in
// flight). Writes
// sel_chunks, sel_groups and n_sel when `write`; with TB == 1 and `s_out`
// given, also leaves the block's selected group ids in s_out[0, top_groups)
// (ascending, -1 padded) and their count in s_out[64] for the caller
// (visible after its next barrier).
template <typename T, int D, int TB, bool EARLY_ROW = true, int RB = 16, typename Sync>
__device__ __forceinline__ void route_blocks(const RouteArgs& a, int wg, bool write, int* s_out, const int tid,
                                             Sync& sync) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E2 = 16 / EB;    // elements per 16-byte slice
  constexpr int SPR = D / E2;    // slices per head row
  extern __shared__ double dyn[];          // phase 0: partial sums [TB][4][D]; then scores [TB][stride]
  __shared__ __attribute__((aligned(16))) double s_q[TB][D];
  __shared__ int s_chunks[TB][64];
  __shared__ int s_ngc[TB];
  __shared__ TopKScratch s_tk[TB];
  __shared__ double s_kv[TB][64];  // rounds: each block's running selection (scores, chunk ids)
  __shared__ int s_ki[TB][64];
  __shared__ int s_part[4][64];  // one block per workgroup: partial ranks of the four waves
  // rounds: the round's candidates that beat a block's running k-th best
  __shared__ double s_sv[TB > 1 ? TB : 1][64];
  __shared__ int s_sf[TB > 1 ? TB : 1][64];
  __shared__ int s_len;

  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = wg % a.n_kv_heads;
  const int b0 = (wg / a.n_kv_heads) * TB;
  const int nb = min(TB, a.n_qb - b0);
  const int64_t qb_abs0 = a.q_begin / 64 + b0;
  const int stride = a.score_stride;

  // candidate chunks of the TB blocks: [c_lo, c_hi)
  const int c_lo = a.first_cand;
  const int c_hi = last_cand(qb_abs0 + nb - 1, a.local_tokens);
  const int n_union = c_hi > c_lo ? c_hi - c_lo : 0;
  // Phase 1 units: (pass of 256 rows, unit of a row). With one block per
  // workgroup (small, latency-bound grids) a row is two halves in two
  // slots, so a pass is one memory round trip; with more blocks (large
  // grids, three waves per SIMD) four quarters in three slots.
  constexpr int UPR = TB == 1 ? 2 : 4;
  constexpr int QPU = D / 4 / UPR;  // summary quads per lane and unit
  // Phases 1-2 run in rounds of RR candidate rows when the host asks for
  // them (a.round_rows > 0, TB > 1 only): the score table then holds one
  // round behind `front` slots for the blocks' running selections.
  const int front = a.round_rows > 0 ? 64 : 0;
  const int RR = a.round_rows > 0 ? a.round_rows : max(n_union, 1);
  const int n_rounds = (n_union + RR - 1) / RR;  // 0 when there are no candidates
  auto round_rows = [&](int r) { return max(0, min(RR, n_union - r * RR)); };
  auto round_units = [&](int r) { return (round_rows(r) + 255) / 256 * UPR; };
  const float* cs = a.chunk_sum + quad_off(h, 0, 0, D, a.chunk_cap);
  // every unit reads an in-bounds row; rows past the round's are not stored
  auto chunk_row = [&](int r, int u) {
    return (int64_t)c_lo + r * RR + min((u / UPR) * 256 + tid, round_rows(r) - 1);
  };
  f32x4 va[QPU], vb[QPU], vc[UPR == 4 ? QPU : 1];  // the register slots of phase 1
  constexpr bool kEarly = EARLY_ROW && TB == 1;  // with TB > 1 the query batches take those registers
  auto first_units = [&](int r) {
    load_unit<D, UPR>(va, cs, chunk_row(r, 0), a.chunk_cap, 0);
    load_unit<D, UPR>(vb, cs, chunk_row(r, 1), a.chunk_cap, 1);
  };
  if constexpr (kEarly) {
    if (n_rounds > 0) first_units(0);
  }

  // ---- phase 0: block descriptors. Thread (sub, col) sums rows sub,
  // sub + nsub, ... of the 16-byte column col of the block's G head rows in
  // float64; the sums of a wave's lanes that hold the same head-dim slice are
  // added across lanes and each wave leaves its partial descriptor in dyn.
  {
    const int G = a.gqa;
    const int cpr = G * SPR;     // slices per block row (G heads), divides 256
    const int nsub = 256 / cpr;  // rows summed in parallel
    const int rows = 64 / nsub;  // rows per thread and block
    const int col = tid % cpr, sub = tid / cpr;
    const int gq = col / SPR, d0 = (col % SPR) * E2;
    const int nbat = (rows + RB - 1) / RB;  // load batches per block
    const int nu = nb * nbat;
    const char* qbase = static_cast<const char*>(a.Q) +
                        ((int64_t)b0 * 64 * a.q_tok + (int64_t)(h * G + gq) * a.q_head + d0) * EB;
    auto load_unit = [&](u32x4 (&raw)[RB], int u) {
      const int t = u / nbat, j0 = (u - t * nbat) * RB;
      const char* base = qbase + (int64_t)t * 64 * a.q_tok * EB;
#pragma unroll
      for (int j = 0; j < RB; ++j) {  // every load in bounds; surplus rows masked in sum_unit
        const int r = sub + nsub * min(j0 + j, rows - 1);
        raw[j] = *reinterpret_cast<const u32x4*>(base + (int64_t)r * a.q_tok * EB);
      }
    };
    double s[E2];
#pragma unroll
    for (int e = 0; e < E2; ++e) s[e] = 0.0;
    auto sum_unit = [&](const u32x4 (&raw)[RB], int u) {
      const int t = u / nbat, j0 = (u - t * nbat) * RB;
#pragma unroll
      for (int j = 0; j < RB; ++j) {
        // surplus loads of a last batch add zero: the row's raw words are
        // cleared under a uniform condition (never, with full batches)
        const u32x4 w = j0 + j < rows ? raw[j] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < E2; ++e) {
          float x;
          if constexpr (EB == 2) x = bf16_bits_to_float((w[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
          else x = __uint_as_float(w[e]);
          s[e] += (double)x;
        }
      }
      if (j0 + RB >= rows) {  // block t summed: fold the wave's lanes of equal slice
#pragma unroll
        for (int e = 0; e < E2; ++e) {
#pragma unroll
          for (int m = SPR; m < 64; m <<= 1) s[e] += shfl_xor_d(s[e], m);
        }
        if (lane < SPR) {
#pragma unroll
          for (int e = 0; e < E2; ++e) dyn[(t * 4 + wave) * D + lane * E2 + e] = s[e];
        }
#pragma unroll
        for (int e = 0; e < E2; ++e) s[e] = 0.0;
      }
    };
    if constexpr (TB == 1) {
#pragma unroll 1
      for (int u = 0; u < nu; ++u) {
        u32x4 raw[RB];
        load_unit(raw, u);
        sum_unit(raw, u);
      }
    } else {
      // two load slots: the next batch is in flight while one is summed. The
      // loads are unconditional (unit indices clamped; a repeated last unit
      // is not summed): conditional ones made the compiler wait for both
      // slots before summing either.
      u32x4 r0[RB], r1[RB];
      load_unit(r0, 0);
#pragma unroll 1
      for (int u = 0; u < nu; u += 2) {
        load_unit(r1, min(u + 1, nu - 1));
        sum_unit(r0, u);
        load_unit(r0, min(u + 2, nu - 1));
        if (u + 1 < nu) sum_unit(r1, u + 1);
      }
    }
    if constexpr (!kEarly) {
      if (n_rounds > 0) first_units(0);
    }
    sync();
    if (tid < D) {
      const double inv = 1.0 / (64.0 * G);
      for (int t = 0; t < nb; ++t) {
        const double* p = dyn + t * 4 * D + tid;
        s_q[t][tid] = ((p[0] + p[D]) + (p[2 * D] + p[3 * D])) * inv;
      }
    }
  }
  sync();

  // ---- phases 1 and 2: chunk scores of every block's candidates (one row
  // per lane, 256 rows per pass), then the top-k_c of each block. With
  // rounds, a block's selection after each round is the top-k_c of its
  // running selection and the round's scores: the kept entries sit ahead of
  // the round's (they have lower chunk indices), so positions keep chunk
  // order and ties still go to the lower index.
  const int gpc_shift = 6 - a.group_shift;  // log2(groups per chunk)
  int n_kept = 0;  // TB > 1: size of this wave's block's running selection
  const int n_loop = TB == 1 ? 1 : max(n_rounds, 1);  // TB == 1: one round, always
#pragma unroll 1
  for (int r = 0; r < n_loop; ++r) {
    const int n_units = round_units(r);
    double a0[TB], a1[TB];
#pragma unroll
    for (int t = 0; t < TB; ++t) a0[t] = a1[t] = 0.0;
    auto consume = [&](f32x4 (&v)[QPU], int u) {
      const int q = u % UPR;
      unit_dots<D, UPR, TB>(v, s_q, q, nb, a0, a1);
      if (q == UPR - 1) {
        const int f = (u / UPR) * 256 + tid;
#pragma unroll
        for (int t = 0; t < TB; ++t) {
          if (t < nb && f < round_rows(r)) dyn[t * stride + front + f] = no_nan(a0[t] + a1[t]);
          a0[t] = a1[t] = 0.0;
        }
      }
    };
    // Slots are named statically at every use and the prefetches inside
    // the loops are unconditional (rows clamped in bounds; the last ones
    // are not consumed): with slots chosen at run time, or conditional
    // loads, the compiler waits for every load in flight.
    if constexpr (UPR == 2) {
      if (n_units == 2) {  // one pass (the usual case): no prefetch beyond it
        consume(va, 0);
        consume(vb, 1);
      } else {
#pragma unroll 1
        for (int u = 0; u < n_units; u += 2) {
          consume(va, u);
          load_unit<D, UPR>(va, cs, chunk_row(r, u + 2), a.chunk_cap, 0);
          consume(vb, u + 1);
          load_unit<D, UPR>(vb, cs, chunk_row(r, u + 3), a.chunk_cap, 1);
        }
      }
    } else {
      // three slots, two units ahead; n_units is a multiple of 4, so one or
      // two units remain after the triples, already loaded
      int u = 0;
#pragma unroll 1
      for (; u + 3 <= n_units; u += 3) {
        load_unit<D, UPR>(vc, cs, chunk_row(r, u + 2), a.chunk_cap, (u + 2) & 3);
        consume(va, u);
        load_unit<D, UPR>(va, cs, chunk_row(r, u + 3), a.chunk_cap, (u + 3) & 3);
        consume(vb, u + 1);
        load_unit<D, UPR>(vb, cs, chunk_row(r, u + 4), a.chunk_cap, (u + 4) & 3);
        consume(vc, u + 2);
      }
      if (u < n_units) consume(va, u);
      if (u + 1 < n_units) consume(vb, u + 1);
    }
    sync();
    if constexpr (TB > 1) {
      // the next round's first units go out ahead of this round's selection
      // (round 0's went out with phase 0; after the last round the last
      // round's rows are requested again and not used)
      if (n_rounds > 0) first_units(min(r + 1, n_rounds - 1));
      // wave t selects for block t over [running selection | this round]
      if (wave < nb) {
        const int t = wave;
        const int n_cand_t = max(0, last_cand(qb_abs0 + t, a.local_tokens) - c_lo);
        const int nr_t = max(0, min(RR, n_cand_t - r * RR));
        if (r == 0 || nr_t > 0) {
          double* base = dyn + t * stride + front - n_kept;
          // Once a block holds k_c chunks, a candidate of this round can only
          // enter its selection by beating the worst of them: it has a higher
          // chunk index than every kept one, so it loses ties, and it must
          // score strictly above the lowest kept score. The few that do are
          // listed after the kept ones and ranked with them; the selection
          // is the one over [kept | whole round].
          const bool pre = r > 0 && n_kept == a.top_chunks;  // the same for every lane
          int n_surv = 0;
          if (pre) {
            double kth = lane < n_kept ? s_kv[t][lane] : __builtin_inf();  // kept in chunk order
#pragma unroll
            for (int m = 1; m < 64; m <<= 1) kth = fmin(kth, shfl_xor_d(kth, m));
            const double* rsc = base + n_kept;  // the round's scores
            for (int f0 = 0; f0 < nr_t; f0 += 64) {
              const int f = f0 + lane;
              const double v = rsc[min(f, nr_t - 1)];
              const bool q = f < nr_t && v > kth;
              const uint64_t m = __ballot(q);
              const int j = n_surv + lanes_below(m);
              if (q && j < 64) {
                s_sv[t][j] = v;
                s_sf[t][j] = f;
              }
              n_surv += __popcll(m);
            }
          }
          const bool listed = pre && n_kept + n_surv <= 64;
          __builtin_amdgcn_wave_barrier();
          if (lane < n_kept) base[lane] = s_kv[t][lane];
          if (listed && lane < n_surv) base[n_kept + lane] = s_sv[t][lane];
          __builtin_amdgcn_wave_barrier();
          const int n = n_kept + (listed ? n_surv : nr_t);
          const int pos = wave_top_k(base, n, a.top_chunks, lane, s_tk[t]);
          const int k_eff = min(a.top_chunks, n);
          double v = 0.0;
          int idx = kNoIdx;
          if (lane < k_eff) {
            v = base[pos];
            idx = pos < n_kept ? s_ki[t][pos]
                               : c_lo + r * RR + (listed ? s_sf[t][pos - n_kept] : pos - n_kept);
          }
          __builtin_amdgcn_wave_barrier();
          if (lane < k_eff) {
            s_kv[t][lane] = v;
            s_ki[t][lane] = idx;
          }
          n_kept = k_eff;
        }
      }
      sync();  // the round's scores are read: the next round may overwrite them
    }
  }

  // the selected chunks of each block, ascending
  {
    const int t = TB == 1 ? 0 : wave;  // this wave's block
    const int64_t slot = (int64_t)(b0 + t) * a.n_kv_heads + h;
    const int n_cand = max(0, last_cand(qb_abs0 + t, a.local_tokens) - c_lo);
    const int kc_eff = min(a.top_chunks, n_cand);
    int chunk = kNoIdx;
    if constexpr (TB == 1) {
      const int pos = block_top_k(dyn, n_cand, a.top_chunks, wave, lane, s_tk[0], s_part, &s_len, sync);
      chunk = pos == kNoIdx ? kNoIdx : c_lo + pos;
    } else if (wave < nb) {
      chunk = lane < n_kept ? s_ki[t][lane] : kNoIdx;
    }
    if (wave < nb) {
      if (write && lane < a.top_chunks) a.sel_chunks[slot * a.top_chunks + lane] = lane < kc_eff ? chunk : -1;
      s_chunks[wave][lane] = chunk;
      if (lane == 0) s_ngc[wave] = kc_eff << gpc_shift;
    }
  }
  sync();

  // ---- phase 3: scores of the chosen chunks' groups; an item is one group
  // of one block. Skipped (a uniform branch) when no chunk can be chosen
  // (top_chunks == 0) or no group is kept (top_groups == 0): nothing reads
  // the scores then, and the item mapping below divides by max_gc.
  const int max_gc = a.top_chunks << gpc_shift;
  if (max_gc > 0 && a.top_groups > 0) {
    const int n_items = nb * max_gc;
    const int gmask = (1 << gpc_shift) - 1;
    const float* gs = a.group_sum + quad_off(h, 0, 0, D, a.group_cap);
    // With a group-summary cache (a.slot_of set), a chunk resident in the
    // cache has its groups read there (rows slot * groups-per-chunk + i),
    // the others from the full table; both hold the same values.
    const float* gcs = a.slot_of ? a.gcache + quad_off(h, 0, 0, D, a.gcache_cap) : gs;
    const int32_t* slot_of = a.slot_of ? a.slot_of + (int64_t)h * a.chunk_cap : nullptr;
    // item f -> (block t, position i, table and row of its group summary);
    // invalid items read row 0 of the full table and get i = -1 (not stored)
    auto group_item = [&](int f, int& t, int& i, const float*& tab, int64_t& cap, int64_t& j) {
      t = min(f / max_gc, nb - 1);
      i = f - t * max_gc;
      const int ch = (f < n_items && i < s_ngc[t]) ? s_chunks[t][i >> gpc_shift] : kNoIdx;
      const bool ok = ch < c_hi;  // always true for the chosen chunks; guards the address
      j = ok ? ((int64_t)ch << gpc_shift) + (i & gmask) : 0;
      tab = gs;
      cap = a.group_cap;
      if (slot_of) {
        const int sl = ok ? slot_of[ch] : -1;
        if (sl >= 0) {
          tab = gcs;
          cap = a.gcache_cap;
          j = ((int64_t)sl << gpc_shift) + (i & gmask);
        }
      }
      if (!ok) i = -1;
    };
    if (a.cache_hit) {
      // hit flag of every chosen chunk: was it resident when the call began
      for (int f = tid; f < n_items; f += 256) {
        const int t = f / max_gc, i = f - t * max_gc;
        if (t < nb && i < s_ngc[t] && (i & gmask) == 0) {
          const int ch = s_chunks[t][i >> gpc_shift];
          a.cache_hit[((int64_t)(b0 + t) * a.n_kv_heads + h) * a.top_chunks + (i >> gpc_shift)] =
              slot_of[ch] >= 0 ? 1 : 0;
        }
      }
    }
    if (n_items <= 64) {
      // Few items (the usual single-block case): lane = item and wave =
      // quarter of its row, so every quarter is in flight at once; the four
      // quarter sums meet in LDS (the selection scratch is free between the
      // two selections) and are added in quarter order.
      int t, i;
      int64_t j, cap;
      const float* tab;
      group_item(lane, t, i, tab, cap, j);
      f32x4 v[D / 16];
      load_unit<D, 4>(v, tab, j, cap, wave);
      double g0[1] = {0.0}, g1[1] = {0.0};
      unit_dots<D, 4, 1>(v, s_q + t, wave, 1, g0, g1);
      double* part = s_tk[0].lv;
      part[wave * 64 + lane] = g0[0] + g1[0];
      sync();
      if (wave == 0 && i >= 0)
        dyn[t * stride + i] = no_nan(((part[lane] + part[64 + lane]) + part[128 + lane]) + part[192 + lane]);
    } else {
      // lane = item as in phase 1, four quarters in three slots
      const int n_units3 = (n_items + 255) / 256 * 4;
      f32x4 ga[D / 16], gb[D / 16], gc[D / 16];
      auto load_g = [&](f32x4 (&v)[D / 16], int u) {
        int t, i;
        int64_t j, cap;
        const float* tab;
        group_item((u >> 2) * 256 + tid, t, i, tab, cap, j);
        load_unit<D, 4>(v, tab, j, cap, u & 3);
      };
      double g0[1] = {0.0}, g1[1] = {0.0};
      auto consume_g = [&](f32x4 (&v)[D / 16], int u) {
        int t, i;
        int64_t j, cap;
        const float* tab;
        group_item((u >> 2) * 256 + tid, t, i, tab, cap, j);
        unit_dots<D, 4, 1>(v, s_q + t, u & 3, 1, g0, g1);
        if ((u & 3) == 3) {
          if (i >= 0) dyn[t * stride + i] = no_nan(g0[0] + g1[0]);
          g0[0] = g1[0] = 0.0;
        }
      };
      load_g(ga, 0);
      load_g(gb, 1);
      int u = 0;
#pragma unroll 1
      for (; u + 3 <= n_units3; u += 3) {  // three static slots, unconditional prefetches
        load_g(gc, u + 2);
        consume_g(ga, u);
        load_g(ga, u + 3);
        consume_g(gb, u + 1);
        load_g(gb, u + 4);
        consume_g(gc, u + 2);
      }
      if (u < n_units3) consume_g(ga, u);
      if (u + 1 < n_units3) consume_g(gb, u + 1);
    }
  }
  sync();

  // ---- phase 4: top-k_g of block `wave` over those groups
  {
    const int t = TB == 1 ? 0 : wave;  // this wave's block
    const int64_t slot = (int64_t)(b0 + t) * a.n_kv_heads + h;
    const int n_gc = s_ngc[t];
    const int kg_eff = min(a.top_groups, n_gc);
    int pos = kNoIdx;
    if (a.top_groups > 0) {
      if constexpr (TB == 1) pos = block_top_k(dyn, n_gc, a.top_groups, wave, lane, s_tk[0], s_part, &s_len, sync);
      else if (wave < nb) pos = wave_top_k(dyn + wave * stride, n_gc, a.top_groups, lane, s_tk[wave]);
    }
    if (wave < nb && a.top_groups > 0) {
      if (lane < a.top_groups) {
        int gid = -1;
        if (lane < kg_eff && pos < n_gc) {
          const int ch = s_chunks[wave][pos >> gpc_shift];
          gid = (ch << gpc_shift) + (pos & ((1 << gpc_shift) - 1));
        }
        if (write) a.sel_groups[slot * a.top_groups + lane] = gid;
        if (TB == 1 && s_out) s_out[lane] = gid;
      }
    }
    if (wave < nb && lane == 0) {
      if (write) a.n_sel[slot] = kg_eff;
      if (TB == 1 && s_out) s_out[64] = kg_eff;
    }
  }
}

}  // namespace hga
