// Routed key set of one (query block, kv head) and the index-driven gather of
// its 64-token tiles into LDS (Sec. 2.1 item 3: only the exact K/V of the
// selected tokens is loaded; summaries are never used as values).
//
// The routed set is laid out as positions [sink | selected groups | local]:
//   sink   : tokens [0, ns),  ns = min(Ws, local start)
//   groups : nsel groups of g tokens, ascending group ids
//   local  : tokens [local start, block end), diagonal block last
// Positions are ascending in token id, every part is disjoint, and the set is
// processed in 64-position tiles; positions >= R are padding (zero rows).
#pragma once
#include "hga_device.h"
#include "hga_kernels.h"

namespace hga {

struct RoutedSet {
  int64_t blk_start;  // first query position of the block
  int64_t local_start;
  int ns;             // sink tokens
  int off;            // first local position
  int R;              // routed set size
  int diag;           // position of token blk_start
  int gshift;
  const int* sel;     // LDS copy of the selected group ids

  __device__ inline int64_t token(int p) const {
    if (p < ns) return p;
    if (p < off) {
      const int q = p - ns;
      return ((int64_t)sel[q >> gshift] << gshift) + (q & ((1 << gshift) - 1));
    }
    if (p < R) return local_start + (p - off);
    return -1;
  }
  // True if some key of positions [p0, p0+64) is masked for a query at
  // offset >= qoff0 within the block (causal or padding).
  __device__ inline bool tile_needs_mask(int p0, int qoff0) const {
    return p0 + 64 > min(R, diag + qoff0 + 1);
  }
  __device__ inline bool masked(int p, int qoff) const { return p >= R || p - diag > qoff; }
};

__device__ inline RoutedSet make_routed_set(const AttnArgs& a, int b, int h, int* s_sel, int tid,
                                            int nthreads) {
  RoutedSet rs;
  rs.blk_start = a.q_begin + (int64_t)b * 64;
  const int64_t blk_end = rs.blk_start + 64;
  rs.local_start = blk_end - a.local_tokens > 0 ? blk_end - a.local_tokens : 0;
  rs.ns = (int)(a.sink_tokens < rs.local_start ? a.sink_tokens : rs.local_start);
  const int64_t slot = (int64_t)b * a.n_kv_heads + h;
  const int nsel = a.n_sel[slot];
  for (int i = tid; i < nsel; i += nthreads) s_sel[i] = a.sel_groups[slot * a.top_groups + i];
  rs.gshift = a.group_shift;
  rs.off = rs.ns + (nsel << a.group_shift);
  rs.R = rs.off + (int)(blk_end - rs.local_start);
  rs.diag = rs.off + (int)(rs.blk_start - rs.local_start);
  rs.sel = s_sel;
  return rs;
}

// Registers holding one thread's share of a 64-token tile of one tensor:
// items are (row pair, 16-byte column) so that a thread owns rows 2rp, 2rp+1.
template <typename T, int D, int NT>
struct TileRegs {
  static constexpr int EB = Elem<T>::kBytes;
  static constexpr int CPR = D * EB / 16;
  static constexpr int NITEMS = 32 * CPR;
  static constexpr int ITEMS = (NITEMS + NT - 1) / NT;
  uint4 r[ITEMS][2];

  __device__ inline void load(const char* base, int64_t tok_stride_b, int64_t head_off_b,
                              const RoutedSet& rs, int tile, int tid) {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int64_t tok = rs.token(tile * 64 + 2 * rp + k);
          if (tok >= 0)
            r[it][k] = *reinterpret_cast<const uint4*>(base + tok * tok_stride_b + head_off_b + cc * 16);
          else
            r[it][k] = make_uint4(0u, 0u, 0u, 0u);
        }
      }
    }
  }

  // Row layout: row = token order within the tile.
  __device__ inline void store_rows(char* dst, int tid) const {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
#pragma unroll
        for (int k = 0; k < 2; ++k)
          *reinterpret_cast<uint4*>(dst + Tile<T, D>::row_off(2 * rp + k, cc * 16 / EB)) = r[it][k];
      }
    }
  }

  // Transposed layout: element (d, kpos_of(row)).
  __device__ inline void store_transposed(char* dst, int tid) const {
    constexpr int E = Elem<T>::E;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
        const uint32_t w0[4] = {r[it][0].x, r[it][0].y, r[it][0].z, r[it][0].w};
        const uint32_t w1[4] = {r[it][1].x, r[it][1].y, r[it][1].z, r[it][1].w};
        if constexpr (EB == 2) {
          const int kp = kpos_of<E>(2 * rp);  // rows 2rp, 2rp+1 sit at kp, kp+1
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const uint32_t lo = (w0[j >> 1] >> ((j & 1) * 16)) & 0xffffu;
            const uint32_t hi = (w1[j >> 1] >> ((j & 1) * 16)) & 0xffffu;
            *reinterpret_cast<uint32_t*>(dst + Tile<T, D>::t_off(cc * 8 + j, kp)) = lo | (hi << 16);
          }
        } else {
          const int kp0 = kpos_of<E>(2 * rp), kp1 = kpos_of<E>(2 * rp + 1);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            *reinterpret_cast<uint32_t*>(dst + Tile<T, D>::t_off(cc * 4 + j, kp0)) = w0[j];
            *reinterpret_cast<uint32_t*>(dst + Tile<T, D>::t_off(cc * 4 + j, kp1)) = w1[j];
          }
        }
      }
    }
  }
};

// Decode a workgroup id into (query block, head slice, kv head). The kv head
// is the fastest index so that consecutive workgroups (dispatched round-robin
// over the 8 XCDs) keep each kv head on one XCD when Hkv == 8, where its
// sink and local-window rows stay in that XCD's L2.
struct WgCoord {
  int b, hs, h;
};
__device__ inline WgCoord decode_wg(int id, int n_kv_heads, int n_hs) {
  WgCoord c;
  c.h = id % n_kv_heads;
  id /= n_kv_heads;
  c.hs = id % n_hs;
  c.b = id / n_hs;
  return c;
}

}  // namespace hga
