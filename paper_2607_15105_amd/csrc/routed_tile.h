// Routed key set of one (query block, kv head) and the index-driven gather of
// its 64-token tiles into LDS (Sec. 2.1 item 3: only the exact K/V of the
// selected tokens is loaded; summaries are never used as values).
//
// The routed set is laid out as positions [sink | local | selected groups]:
//   sink   : tokens [0, ns),  ns = min(Ws, local start)
//   local  : tokens [local start, block end), diagonal block last
//   groups : nsel groups of g tokens, ascending group ids
// Every part is disjoint and the set is processed in 64-position tiles;
// positions >= R are padding (zero rows). Ws, Wl and the block are multiples
// of 64, so the window positions [0, nw) fill whole tiles that are known
// before the routing is: they can be gathered, and attended, while the
// block's routing is still being computed.
#pragma once
#include "hga_device.h"
#include "hga_kernels.h"

namespace hga {

struct RoutedSet {
  int64_t blk_start;  // first query position of the block
  int64_t local_start;
  int ns;             // sink tokens
  int nw;             // window positions (sink + local), a multiple of 64
  int R;              // routed set size
  int diag;           // position of token blk_start (first of the diagonal tile)
  int gshift;
  const int* sel;     // LDS copy of the selected group ids

  // First token of window tile w (w < nw / 64): 64 consecutive tokens.
  __device__ inline int64_t window_first(int w) const {
    const int p0 = 64 * w;
    return p0 < ns ? (int64_t)p0 : local_start + (p0 - ns);
  }
  // Token of position p, computed without branches. Positions past the
  // routed set (padding) return the block's first token, a row that exists,
  // and report ok = false so the caller zeroes what it loaded.
  __device__ inline int64_t token(int p, bool& ok) const {
    const int q = p - nw;
    const int qmax = R - nw - 1;
    const int qi = q < 0 ? 0 : (q > qmax ? (qmax > 0 ? qmax : 0) : q);
    const int64_t tg = ((int64_t)sel[qi >> gshift] << gshift) + (qi & ((1 << gshift) - 1));
    const int64_t tw = p < ns ? (int64_t)p : local_start + (p - ns);
    const int64_t t = p < nw ? tw : tg;
    ok = p < R;
    return ok ? t : blk_start;
  }
  // Token of position p in the selected-group part (p >= nw; the caller
  // knows the whole tile lies there). Padding positions (p >= R) return the
  // first selected token, which exists whenever a group tile does.
  __device__ inline int64_t group_token(int p, bool& ok) const {
    ok = p < R;
    const int qi = ok ? p - nw : 0;
    return ((int64_t)sel[qi >> gshift] << gshift) + (qi & ((1 << gshift) - 1));
  }
  // True if some key of positions [p0, p0+64) is masked for a query at
  // offset >= qoff0 within the block: padding, or the diagonal tile's keys
  // after the query (only that tile holds tokens of the block itself).
  __device__ inline bool tile_needs_mask(int p0, int qoff0) const {
    return p0 + 64 > R || (p0 < diag + 64 && p0 + 64 > diag + qoff0 + 1);
  }
  __device__ inline bool masked(int p, int qoff) const {
    return p >= R || (p - diag > qoff && p < diag + 64);
  }
};

// The window part of block b's routed set (everything but the selected
// groups): usable before the routing row is known, for window tiles only.
// `sel` is the LDS array that will hold the selected group ids: token() may
// read it (and discard what it reads) before it is filled.
__device__ inline RoutedSet window_set(const AttnArgs& a, int b, const int* sel) {
  RoutedSet rs;
  rs.blk_start = a.q_begin + (int64_t)b * 64;
  const int64_t blk_end = rs.blk_start + 64;
  rs.local_start = blk_end - a.local_tokens > 0 ? blk_end - a.local_tokens : 0;
  rs.ns = (int)(a.sink_tokens < rs.local_start ? a.sink_tokens : rs.local_start);
  rs.nw = rs.ns + (int)(blk_end - rs.local_start);
  rs.diag = rs.nw - 64;
  rs.gshift = a.group_shift;
  rs.R = rs.nw;
  rs.sel = sel;
  return rs;
}

// Completes a window set with the block's routing: nsel selected groups whose
// ids are sel[0, nsel) (an LDS array, ascending).
__device__ inline void set_groups(RoutedSet& rs, int nsel, const int* sel) {
  rs.R = rs.nw + (nsel << rs.gshift);
  rs.sel = sel;
}

// The routing row of (block b, kv head h): the selected-group count and,
// for threads below top_groups, one entry of the row (padding entries are
// -1 and never read back). Issued before anything else a kernel loads so
// that the gather addresses are known after one memory round trip.
struct RouteRow {
  int nsel;
  int sel;
};

__device__ inline RouteRow load_route_row(const AttnArgs& a, int b, int h, int tid) {
  const int64_t slot = (int64_t)b * a.n_kv_heads + h;
  RouteRow r;
  r.nsel = a.n_sel[slot];
  r.sel = tid < a.top_groups ? a.sel_groups[slot * a.top_groups + tid] : -1;
  return r;
}

// Routed set of block b from its routing row; the selected group ids go to
// s_sel (the caller synchronizes before the first token() call). Needs at
// least top_groups (<= 64) threads.
__device__ inline RoutedSet make_routed_set(const AttnArgs& a, int b, const RouteRow& row,
                                            int* s_sel, int tid) {
  RoutedSet rs = window_set(a, b, s_sel);
  if (tid < a.top_groups) s_sel[tid] = row.sel;
  set_groups(rs, row.nsel, s_sel);
  return rs;
}

// Registers holding one thread's share of a 64-token tile of K and V:
// items are (row pair, 16-byte column) so that a thread owns rows 2rp, 2rp+1
// of both tensors. Every load is unconditional (padding rows read a real row),
// so a tile's loads are all in flight together. ZP: padding rows are zeroed
// when stored; without it they are stored as loaded, for consumers that mask
// every padding key's score to -inf (its probability is then exactly zero
// and the finite row it holds never reaches an output).
template <typename T, int D, int NT, bool ZP = true>
struct KVRegs {
  static constexpr int EB = Elem<T>::kBytes;
  static constexpr int CPR = D * EB / 16;
  static constexpr int NITEMS = 32 * CPR;
  static constexpr int ITEMS = (NITEMS + NT - 1) / NT;
  uint4 k[ITEMS][2], v[ITEMS][2];
  uint32_t valid;  // bit 2*it + r: row r of item it is inside the routed set

  __device__ inline void load(const char* kb, int64_t k_tok_b, const char* vb, int64_t v_tok_b,
                              const RoutedSet& rs, int tile, int tid) {
    valid = 0;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          bool ok;
          const int64_t tok = rs.token(tile * 64 + 2 * rp + r, ok);
          valid |= (uint32_t)ok << (2 * it + r);
          k[it][r] = *reinterpret_cast<const uint4*>(row_ptr(kb, tok, k_tok_b) + cc * 16);
          v[it][r] = *reinterpret_cast<const uint4*>(row_ptr(vb, tok, v_tok_b) + cc * 16);
        }
      }
    }
  }

  // A tile of the selected-group part (64 * tile >= rs.nw). Rows 2rp and
  // 2rp + 1 are consecutive tokens of one group when groups have two or more
  // tokens (g and the window part are even), so one lookup serves both.
  __device__ inline void load_groups(const char* kb, int64_t k_tok_b, const char* vb, int64_t v_tok_b,
                                     const RoutedSet& rs, int tile, int tid) {
    valid = 0;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
        bool ok0, ok1;
        const int64_t t0 = rs.group_token(tile * 64 + 2 * rp, ok0);
        int64_t t1;
        if (rs.gshift > 0) {
          t1 = t0 + 1;
          ok1 = ok0;
        } else {
          t1 = rs.group_token(tile * 64 + 2 * rp + 1, ok1);
        }
        if constexpr (ZP) valid |= ((uint32_t)ok0 << (2 * it)) | ((uint32_t)ok1 << (2 * it + 1));
        k[it][0] = *reinterpret_cast<const uint4*>(row_ptr(kb, t0, k_tok_b) + cc * 16);
        v[it][0] = *reinterpret_cast<const uint4*>(row_ptr(vb, t0, v_tok_b) + cc * 16);
        k[it][1] = *reinterpret_cast<const uint4*>(row_ptr(kb, t1, k_tok_b) + cc * 16);
        v[it][1] = *reinterpret_cast<const uint4*>(row_ptr(vb, t1, v_tok_b) + cc * 16);
      }
    }
  }

  // 64 consecutive tokens from `first` (a window tile): no routing
  // information needed, so it can be issued before the routing is known.
  __device__ inline void load_contiguous(const char* kb, int64_t k_tok_b, const char* vb, int64_t v_tok_b,
                                         int64_t first, int tid) {
    valid = ~0u;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int64_t tok = first + 2 * rp + r;
          k[it][r] = *reinterpret_cast<const uint4*>(row_ptr(kb, tok, k_tok_b) + cc * 16);
          v[it][r] = *reinterpret_cast<const uint4*>(row_ptr(vb, tok, v_tok_b) + cc * 16);
        }
      }
    }
  }

  __device__ inline uint4 get(const uint4 (&x)[ITEMS][2], int it, int r) const {
    if constexpr (!ZP) return x[it][r];
    return ((valid >> (2 * it + r)) & 1u) ? x[it][r] : make_uint4(0u, 0u, 0u, 0u);
  }

  // Rows 64 tile + (0..63) of a compact [rows][D] copy at kdst / vdst (row
  // pitch D elements); padding rows are written as zeros.
  __device__ inline void store_global(char* kdst, char* vdst, int tile, int tid) const {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int64_t off = ((int64_t)tile * 64 + 2 * rp + r) * (D * EB) + cc * 16;
          *reinterpret_cast<uint4*>(kdst + off) = get(k, it, r);
          *reinterpret_cast<uint4*>(vdst + off) = get(v, it, r);
        }
      }
    }
  }

  // Row layout: row = position within the tile.
  __device__ inline void store_rows(char* dst, bool of_v, int tid) const {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
#pragma unroll
        for (int r = 0; r < 2; ++r)
          *reinterpret_cast<uint4*>(dst + Tile<T, D>::row_off(2 * rp + r, cc * 16 / EB)) =
              get(of_v ? v : k, it, r);
      }
    }
  }

  // Transposed layout: element (d, kpos_of(row)).
  __device__ inline void store_transposed(char* dst, bool of_v, int tid) const {
    constexpr int E = Elem<T>::E;
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int item = tid + it * NT;
      if (NITEMS % NT == 0 || item < NITEMS) {
        const int rp = item / CPR, cc = item % CPR;
        const uint4 a0 = get(of_v ? v : k, it, 0), a1 = get(of_v ? v : k, it, 1);
        const uint32_t w0[4] = {a0.x, a0.y, a0.z, a0.w};
        const uint32_t w1[4] = {a1.x, a1.y, a1.z, a1.w};
        if constexpr (EB == 2) {
          const int kp = kpos_of<E>(2 * rp);  // rows 2rp, 2rp+1 sit at kp, kp+1
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            // low halves (even j) or high halves (odd j) of the two rows' words
            const uint32_t pk = __builtin_amdgcn_perm(w1[j >> 1], w0[j >> 1],
                                                      (j & 1) ? 0x07060302u : 0x05040100u);
            *reinterpret_cast<uint32_t*>(dst + Tile<T, D>::t_off(cc * 8 + j, kp)) = pk;
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
