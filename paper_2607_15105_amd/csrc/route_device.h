// Two-level routing (Sec. 2.1 items 1-2, Fig. 1), device code shared by the
// routing kernel and the fused routing + forward kernel. A workgroup of four
// waves handles TB consecutive query blocks of one kv head:
//
//   phase 0  block descriptor qbar = mean of the block's B rows over the G
//            query heads of the kv head, summed exactly in float64 (bf16 has
//            8 significant bits) and scaled by 1/(B*G), a power of two;
//   phase 1  chunk scores qbar . s^C for every candidate chunk of the TB
//            blocks. Lane = chunk: a lane loads its whole summary row at once,
//            so one memory round trip serves the row, and scores it against
//            all TB descriptors (each row is read once per workgroup);
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

// float64 score of one summary row (D floats, loaded whole) against q, as
// CH interleaved FMA chains over the head dim (d mod CH) summed at the end:
// more chains shorten the dependent latency, fewer keep registers low.
template <int D, int CH>
__device__ inline double score_row(f32x4 (&v)[D / 4], const double* q) {
  double acc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) acc[c] = 0.0;
#pragma unroll
  for (int j = 0; j < D / 4; ++j) {
    // work in groups of 16 values: the descriptor reads and the row's
    // conversions to double of a group are not moved ahead of it, so they
    // never hold more than a group's registers
    if (j % 4 == 0) {
      asm volatile("" ::: "memory");
#pragma unroll
      for (int u = 0; u < 4; ++u) asm volatile("" : "+v"(v[j + u]));
    }
    const double2 q01 = *reinterpret_cast<const double2*>(q + 4 * j);
    const double2 q23 = *reinterpret_cast<const double2*>(q + 4 * j + 2);
    acc[0 % CH] = fma((double)v[j][0], q01.x, acc[0 % CH]);
    acc[1 % CH] = fma((double)v[j][1], q01.y, acc[1 % CH]);
    acc[2 % CH] = fma((double)v[j][2], q23.x, acc[2 % CH]);
    acc[3 % CH] = fma((double)v[j][3], q23.y, acc[3 % CH]);
  }
  if constexpr (CH == 4) return (acc[0] + acc[1]) + (acc[2] + acc[3]);
  else return acc[0];
}

// Row r of a summary table of one kv head (quad-major, `cap` rows): quad j of
// the row sits cap quads after quad j - 1, so lanes reading consecutive rows
// read consecutive 16-byte quads.
template <int D>
__device__ inline void load_row(f32x4 (&v)[D / 4], const float* table, int64_t r, int64_t cap) {
  const f32x4* t = reinterpret_cast<const f32x4*>(table) + r;
#pragma unroll
  for (int j = 0; j < D / 4; ++j) v[j] = t[j * cap];
}

// Routing of the TB query blocks of workgroup `wg` on four waves whose thread
// ids are `tid` (0..255) and whose barrier is `sync`, in the phases
// described at the top; RB query-row loads are in flight per thread in
// phase 0 (EARLY_ROW: see v0 below). Writes sel_chunks, sel_groups and n_sel when
// `write`; with TB == 1 and `s_out` given, also leaves the block's selected
// group ids in s_out[0, top_groups) (ascending, -1 padded) and their count in
// s_out[64] for the caller (visible after its next barrier).
template <typename T, int D, int TB, bool EARLY_ROW = true, int RB = 16, typename Sync>
__device__ __forceinline__ void route_blocks(const RouteArgs& a, int wg, bool write, int* s_out, const int tid,
                                             Sync& sync) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E2 = 16 / EB;    // elements per 16-byte slice
  constexpr int SPR = D / E2;    // slices per head row
  constexpr int SCH = TB == 1 ? 4 : 1;  // FMA chains per score
  extern __shared__ double dyn[];          // phase 0: sums; then scores [TB][stride]
  __shared__ __attribute__((aligned(16))) double s_q[TB][D];
  __shared__ int s_chunks[TB][64];
  __shared__ int s_ngc[TB];
  __shared__ TopKScratch s_tk[4];
  __shared__ int s_part[4][64];  // one block per workgroup: partial ranks of the four waves
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
  const float* cs = a.chunk_sum + quad_off(h, 0, 0, D, a.chunk_cap);
  // With one block per workgroup (small grids, latency-bound) the first
  // summary row of each thread is requested early, so that its memory round
  // trip overlaps the descriptor's: before the query rows (EARLY_ROW), or
  // once they have been summed, ahead of the cross-thread reduction (which
  // keeps the row's registers free while the query rows are in flight).
  f32x4 v0[TB == 1 ? D / 4 : 1];
  if constexpr (TB == 1 && EARLY_ROW) {
    if (tid < n_union) load_row<D>(v0, cs, c_lo + tid, a.chunk_cap);
  }

  // ---- phase 0: block descriptors
  {
    const int G = a.gqa;
    const int cpr = G * SPR;     // slices per block row (G heads), divides 256
    const int nsub = 256 / cpr;  // rows summed in parallel
    const int rows = 64 / nsub;  // rows per thread
    const int col = tid % cpr, sub = tid / cpr;
    const int gq = col / SPR, d0 = (col % SPR) * E2;
    const double inv = 1.0 / (64.0 * G);
#pragma unroll 1
    for (int t = 0; t < nb; ++t) {
      const char* base = static_cast<const char*>(a.Q) +
                         ((int64_t)(b0 + t) * 64 * a.q_tok + (int64_t)(h * G + gq) * a.q_head + d0) * EB;
      double s[E2];
#pragma unroll
      for (int e = 0; e < E2; ++e) s[e] = 0.0;
      for (int j0 = 0; j0 < rows; j0 += RB) {
        u32x4 raw[RB];
#pragma unroll
        for (int j = 0; j < RB; ++j) {  // every load in bounds; surplus rows masked below
          const int r = sub + nsub * min(j0 + j, rows - 1);
          raw[j] = *reinterpret_cast<const u32x4*>(base + (int64_t)r * a.q_tok * EB);
        }
#pragma unroll
        for (int j = 0; j < RB; ++j) {
          if (j0 + j < rows) {
#pragma unroll
            for (int e = 0; e < E2; ++e) {
              float x;
              if constexpr (EB == 2) x = bf16_bits_to_float((raw[j][e >> 1] >> ((e & 1) * 16)) & 0xffffu);
              else x = __uint_as_float(raw[j][e]);
              s[e] += (double)x;
            }
          }
        }
      }
      if constexpr (TB == 1 && !EARLY_ROW) {
        if (tid < n_union) load_row<D>(v0, cs, c_lo + tid, a.chunk_cap);
      }
      sync();  // dyn free
#pragma unroll
      for (int e = 0; e < E2; ++e) dyn[tid * E2 + e] = s[e];
      sync();
      if (tid < D) {
        const int cd = tid / E2, ed = tid % E2;
        double tot = 0.0;
        for (int g2 = 0; g2 < G; ++g2)
          for (int sb = 0; sb < nsub; ++sb) tot += dyn[(sb * cpr + g2 * SPR + cd) * E2 + ed];
        s_q[t][tid] = tot * inv;
      }
    }
  }
  sync();

  // ---- phase 1: chunk scores of every block's candidates
  if constexpr (TB == 1) {
    if (tid < n_union) dyn[tid] = no_nan(score_row<D, SCH>(v0, s_q[0]));
  }
  for (int i = tid + (TB == 1 ? 256 : 0); i < n_union; i += 256) {
    // keep the descriptor reads inside the loop (hoisted, they would hold
    // TB x D doubles in registers)
    asm volatile("" ::: "memory");
    f32x4 v[D / 4];
    load_row<D>(v, cs, c_lo + i, a.chunk_cap);
#pragma unroll 1
    for (int t = 0; t < nb; ++t) {
      // the row stays float: its conversion to double is not hoisted out of
      // this loop (that would hold 2 x D registers)
#pragma unroll
      for (int j = 0; j < D / 4; ++j) asm volatile("" : "+v"(v[j]));
      dyn[t * stride + i] = no_nan(score_row<D, SCH>(v, s_q[t]));
    }
  }
  sync();

  // ---- phase 2: top-k_c of block `wave`
  const int gpc_shift = 6 - a.group_shift;  // log2(groups per chunk)
  {
    const int t = TB == 1 ? 0 : wave;  // this wave's block
    const int64_t slot = (int64_t)(b0 + t) * a.n_kv_heads + h;
    const int n_cand = max(0, last_cand(qb_abs0 + t, a.local_tokens) - c_lo);
    const int kc_eff = min(a.top_chunks, n_cand);
    int pos = kNoIdx;
    if constexpr (TB == 1) pos = block_top_k(dyn, n_cand, a.top_chunks, wave, lane, s_tk[0], s_part, &s_len, sync);
    else if (wave < nb) pos = wave_top_k(dyn + wave * stride, n_cand, a.top_chunks, lane, s_tk[wave]);
    if (wave < nb) {
    const int chunk = pos == kNoIdx ? kNoIdx : c_lo + pos;
    if (write && lane < a.top_chunks) a.sel_chunks[slot * a.top_chunks + lane] = lane < kc_eff ? chunk : -1;
    s_chunks[wave][lane] = chunk;
    if (lane == 0) s_ngc[wave] = kc_eff << gpc_shift;
    }
  }
  sync();

  // ---- phase 3: scores of the chosen chunks' groups
  const int max_gc = a.top_chunks << gpc_shift;
  const float* gs = a.group_sum + quad_off(h, 0, 0, D, a.group_cap);
  for (int f = tid; f < nb * max_gc; f += 256) {
    asm volatile("" ::: "memory");
    const int t = f / max_gc, i = f - t * max_gc;
    const int ch = i < s_ngc[t] ? s_chunks[t][i >> gpc_shift] : kNoIdx;
    if (ch < c_hi) {  // always true for the chosen chunks; guards the address
      const int64_t j = ((int64_t)ch << gpc_shift) + (i & ((1 << gpc_shift) - 1));
      f32x4 v[D / 4];
      load_row<D>(v, gs, j, a.group_cap);
      dyn[t * stride + i] = no_nan(score_row<D, SCH>(v, s_q[t]));
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
