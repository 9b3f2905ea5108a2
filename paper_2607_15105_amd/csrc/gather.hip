// The exact-token gather of Sec. 2.1 item 3 as a kernel of its own: the K/V
// rows of every (query block, kv head)'s routed set, in the attention
// kernels' tile order [sink | local | selected groups], copied to compact
// buffers [n_qb][Hkv][r_cap][D]. The attention kernels do the same gather
// into LDS tiles without this copy; this kernel exists to measure the
// gather's bandwidth apart from the attention (and to feed the forward over
// compact rows, which isolates the attention tiles).
//
// One workgroup of 256 threads per (block, kv head); two register slots keep
// two tiles' loads in flight while the previous tile is stored. Every load
// and store is a 16-byte piece of a row: loads hit one routed row per
// (row pair, piece) item, stores are contiguous 16 KB tiles.
#include "routed_tile.h"

namespace hga {

template <typename T, int D>
__global__ __launch_bounds__(256) void gather_kernel(AttnArgs a, char* kc, char* vc) {
  constexpr int EB = Elem<T>::kBytes;
  __shared__ int s_sel[64];
  const int tid = threadIdx.x;
  const int h = blockIdx.x % a.n_kv_heads, b = blockIdx.x / a.n_kv_heads;
  const RouteRow rrow = load_route_row(a, b, h, tid);
  const RoutedSet rs = make_routed_set(a, b, rrow, s_sel, tid);
  __syncthreads();  // s_sel
  const int ntiles = (rs.R + 63) >> 6;
  const char* kb = static_cast<const char*>(a.K) + (int64_t)h * a.k_head * EB;
  const char* vb = static_cast<const char*>(a.V) + (int64_t)h * a.v_head * EB;
  const int64_t ktb = a.k_tok * EB, vtb = a.v_tok * EB;
  const int64_t slot = ((int64_t)b * a.n_kv_heads + h) * a.r_cap * D * EB;
  char* kd = kc + slot;
  char* vd = vc + slot;
  KVRegs<T, D, 256> r0, r1;
  r0.load(kb, ktb, vb, vtb, rs, 0, tid);
  if (ntiles > 1) r1.load(kb, ktb, vb, vtb, rs, 1, tid);
  for (int t = 0; t < ntiles; t += 2) {
    r0.store_global(kd, vd, t, tid);
    if (t + 2 < ntiles) r0.load(kb, ktb, vb, vtb, rs, t + 2, tid);
    if (t + 1 < ntiles) {
      r1.store_global(kd, vd, t + 1, tid);
      if (t + 3 < ntiles) r1.load(kb, ktb, vb, vtb, rs, t + 3, tid);
    }
  }
}

hipError_t launch_gather(const AttnArgs& a, void* kc, void* vc, bool bf16, int head_dim, hipStream_t s) {
  const dim3 grid(a.n_qb * a.n_kv_heads);
  char* k = static_cast<char*>(kc);
  char* v = static_cast<char*>(vc);
  if (bf16) {
    if (head_dim == 64) hipLaunchKernelGGL((gather_kernel<__bf16, 64>), grid, dim3(256), 0, s, a, k, v);
    else hipLaunchKernelGGL((gather_kernel<__bf16, 128>), grid, dim3(256), 0, s, a, k, v);
  } else {
    hipLaunchKernelGGL((gather_kernel<float, 64>), grid, dim3(256), 0, s, a, k, v);  // float32: head_dim 64
  }
  return hipGetLastError();
}

}  // namespace hga
