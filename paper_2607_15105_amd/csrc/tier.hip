// Tiered storage (Sec. 2.2, Fig. 2; Sec. 2.1 item 2): history K/V and the
// full table of group summaries live in host RAM, the chunk summaries and a
// bounded cache of group summaries in device memory, and the exact K/V rows
// a call routes to are staged into a compact routed working set in device
// memory before attention runs over it.
//
//   cache_clear_kernel   empties a cache (no slot holds a chunk);
//   cache_update_kernel  after a routing call: the chunks the call chose that
//                        were not resident are brought in, first-in
//                        first-out, in ascending chunk order, evicting the
//                        oldest slots (one workgroup per kv head). The order
//                        depends only on the call's routing, so the cache's
//                        contents and every later hit are reproducible;
//   tier_gather_kernel   the routed rows of every (block, kv head), history
//                        rows read from host memory over the bus and active
//                        rows from device memory, into compact rows.
//
// Host memory is read and written through its device-mapped address; the
// kernels see no difference other than the bus.
#include "routed_tile.h"

namespace hga {

__global__ __launch_bounds__(256) void cache_clear_kernel(CacheArgs c) {
  const int64_t n_map = (int64_t)c.n_kv_heads * c.chunk_cap;
  const int64_t n_slot = (int64_t)c.n_kv_heads * c.n_slots;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_map + n_slot + c.n_kv_heads; i += stride) {
    if (i < n_map) c.slot_of[i] = -1;
    else if (i < n_map + n_slot) c.slot_chunk[i - n_map] = -1;
    else c.cursor[i - n_map - n_slot] = 0;
  }
}

template <int D>
__global__ __launch_bounds__(256) void cache_update_kernel(CacheArgs c) {
  extern __shared__ uint32_t s_bits[];  // missed chunks of the call, one bit each
  __shared__ int s_part[256];
  __shared__ int s_ins[kMaxCacheSlots];  // chunk inserted k-th (k < n_ins)
  __shared__ int s_total;
  const int tid = threadIdx.x;
  const int h = blockIdx.x;
  const int nw = (int)((c.chunk_cap + 31) / 32);
  for (int w = tid; w < nw; w += 256) s_bits[w] = 0u;
  __syncthreads();
  const int64_t n_ent = (int64_t)c.n_qb * c.top_chunks;
  for (int64_t e = tid; e < n_ent; e += 256) {
    const int64_t b = e / c.top_chunks, r = e % c.top_chunks;
    const int64_t at = (b * c.n_kv_heads + h) * c.top_chunks + r;
    const int ch = c.sel_chunks[at];
    if (ch >= 0 && c.cache_hit[at] == 0) atomicOr(&s_bits[ch >> 5], 1u << (ch & 31));
  }
  __syncthreads();
  // rank of every missed chunk in ascending order: words are split into 256
  // contiguous runs, one per thread
  const int per = (nw + 255) / 256;
  const int w0 = min(nw, tid * per), w1 = min(nw, w0 + per);
  int cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(s_bits[w]);
  s_part[tid] = cnt;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int i = 0; i < 256; ++i) {
      const int x = s_part[i];
      s_part[i] = run;
      run += x;
    }
    s_total = run;
  }
  __syncthreads();
  const int M = s_total;
  const int S = (int)c.n_slots;
  const int n_ins = min(M, S);  // the last S misses stay (earlier ones would be evicted by later ones)
  const int first = M - n_ins;
  const int cur = c.cursor[h];
  int32_t* slot_of = c.slot_of + (int64_t)h * c.chunk_cap;
  int32_t* slot_chunk = c.slot_chunk + (int64_t)h * c.n_slots;
  // evictions first: the slots about to be filled release their chunks
  for (int k = tid; k < n_ins; k += 256) {
    const int old = slot_chunk[(cur + k) % S];
    if (old >= 0) slot_of[old] = -1;
  }
  __syncthreads();
  int rank = s_part[tid];
  for (int w = w0; w < w1; ++w) {
    uint32_t m = s_bits[w];
    while (m) {
      const int bit = __ffs(m) - 1;
      m &= m - 1;
      if (rank >= first) {
        const int ch = w * 32 + bit;
        const int slot = (cur + rank - first) % S;
        slot_chunk[slot] = ch;
        slot_of[ch] = slot;
        s_ins[rank - first] = ch;
      }
      ++rank;
    }
  }
  __syncthreads();
  // copy the inserted chunks' group summaries into their slots (quad-major:
  // the gpc groups of a chunk are gpc consecutive 16-byte entries per quad)
  const int gpc = 1 << c.gpc_shift;
  const int64_t items = (int64_t)n_ins * (D / 4) * gpc;
  // eight 16-byte pieces in flight per thread: the table is read over the
  // host link, where one piece at a time would wait a round trip each
  constexpr int U = 8;
  for (int64_t it0 = tid; it0 < items; it0 += 256 * U) {
    f32x4 v[U];
    int64_t dst[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t it = min(it0 + 256 * u, items - 1);  // past the end: the last piece again, not stored
      const int i = (int)(it % gpc);
      const int q = (int)((it / gpc) % (D / 4));
      const int k = (int)(it / ((int64_t)gpc * (D / 4)));
      const int ch = s_ins[k];
      v[u] = *reinterpret_cast<const f32x4*>(
          c.group_sum + quad_off(h, q, ((int64_t)ch << c.gpc_shift) + i, D, c.group_cap));
      dst[u] = quad_off(h, q, ((int64_t)((cur + k) % S) << c.gpc_shift) + i, D, (int64_t)S << c.gpc_shift);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (it0 + 256 * u < items) *reinterpret_cast<f32x4*>(c.groups + dst[u]) = v[u];
  }
  if (tid == 0) c.cursor[h] = (cur + n_ins) % S;
}

size_t cache_update_lds_bytes(int64_t chunk_cap) { return (size_t)((chunk_cap + 31) / 32) * 4; }

hipError_t launch_cache_clear(const CacheArgs& c, hipStream_t s) {
  const int64_t n = (int64_t)c.n_kv_heads * (c.chunk_cap + c.n_slots + 1);
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(cache_clear_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, s, c);
  return hipGetLastError();
}

hipError_t launch_cache_update(const CacheArgs& c, int head_dim, hipStream_t s) {
  const size_t lds = cache_update_lds_bytes(c.chunk_cap);
  if (head_dim == 64) hipLaunchKernelGGL((cache_update_kernel<64>), dim3(c.n_kv_heads), dim3(256), lds, s, c);
  else hipLaunchKernelGGL((cache_update_kernel<128>), dim3(c.n_kv_heads), dim3(256), lds, s, c);
  return hipGetLastError();
}

// ---------------------------------------------------------------- gather

// Row `tok` of a K or V tensor split at hist_end: history rows from the host
// copy, the others from the device copy whose row 0 is token hist_end.
__device__ inline const char* tier_row(const char* hist, int64_t h_tok_b, const char* act, int64_t a_tok_b,
                                       int64_t hist_end, int64_t tok) {
  return tok < hist_end ? row_ptr(hist, tok, h_tok_b) : row_ptr(act, tok - hist_end, a_tok_b);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void tier_gather_kernel(AttnArgs a, TierArgs t, char* kc, char* vc) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int CPR = D * EB / 16;        // 16-byte pieces per row
  constexpr int PER = 64 * CPR / 256;     // pieces per thread and tile
  __shared__ int s_sel[64];
  const int tid = threadIdx.x;
  const int h = blockIdx.x % a.n_kv_heads, b = blockIdx.x / a.n_kv_heads;
  const RouteRow rrow = load_route_row(a, b, h, tid);
  const RoutedSet rs = make_routed_set(a, b, rrow, s_sel, tid);
  __syncthreads();  // s_sel
  const int ntiles = (rs.R + 63) >> 6;
  const char* kh = static_cast<const char*>(t.K_hist) + (int64_t)h * t.h_head * EB;
  const char* vh = static_cast<const char*>(t.V_hist) + (int64_t)h * t.h_head * EB;
  const char* ka = static_cast<const char*>(t.K_act) + (int64_t)h * t.a_head * EB;
  const char* va = static_cast<const char*>(t.V_act) + (int64_t)h * t.a_head * EB;
  const int64_t htb = t.h_tok * EB, atb = t.a_tok * EB;
  const int64_t slot = ((int64_t)b * a.n_kv_heads + h) * a.r_cap * D * EB;
  for (int tile = 0; tile < ntiles; ++tile) {
    uint4 kx[PER], vx[PER];
    bool ok[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {  // every load of the tile in flight together
      const int item = tid + 256 * u;
      const int r = item / CPR, cc = item % CPR;
      const int64_t tok = rs.token(tile * 64 + r, ok[u]);
      kx[u] = *reinterpret_cast<const uint4*>(tier_row(kh, htb, ka, atb, t.hist_end, tok) + cc * 16);
      vx[u] = *reinterpret_cast<const uint4*>(tier_row(vh, htb, va, atb, t.hist_end, tok) + cc * 16);
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int item = tid + 256 * u;
      const int r = item / CPR, cc = item % CPR;
      const int64_t off = slot + ((int64_t)tile * 64 + r) * (D * EB) + cc * 16;
      *reinterpret_cast<uint4*>(kc + off) = ok[u] ? kx[u] : make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(vc + off) = ok[u] ? vx[u] : make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

hipError_t launch_tier_gather(const AttnArgs& a, const TierArgs& t, void* kc, void* vc, bool bf16, int head_dim,
                              hipStream_t s) {
  const dim3 grid(a.n_qb * a.n_kv_heads);
  char* k = static_cast<char*>(kc);
  char* v = static_cast<char*>(vc);
  if (bf16) {
    if (head_dim == 64) hipLaunchKernelGGL((tier_gather_kernel<__bf16, 64>), grid, dim3(256), 0, s, a, t, k, v);
    else hipLaunchKernelGGL((tier_gather_kernel<__bf16, 128>), grid, dim3(256), 0, s, a, t, k, v);
  } else {
    hipLaunchKernelGGL((tier_gather_kernel<float, 64>), grid, dim3(256), 0, s, a, t, k, v);
  }
  return hipGetLastError();
}

}  // namespace hga
