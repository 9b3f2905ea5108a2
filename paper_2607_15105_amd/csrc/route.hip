// Routing kernel (Sec. 2.1 items 1-2): one launch routes every query block
// of a call; the phases are the device code of route_device.h.
#include "route_device.h"

namespace hga {

// Several blocks per workgroup (large grids): three waves per SIMD, since
// the scoring passes are latency-bound and the register budget that allows
// (168) holds their three prefetch slots. One block (small grids, one
// workgroup per CU): the register budget goes to a pass's two half rows.
template <typename T, int D, int TB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(TB == 1 ? 1 : 3))) void route_kernel(RouteArgs a) {
  prefetch_args(a);
  WgSync sync;
  route_blocks<T, D, TB, true, TB == 1 ? 16 : 8>(a, blockIdx.x, true, nullptr, (int)threadIdx.x, sync);
}

size_t route_lds_bytes(int tb, int score_stride, bool bf16) {
  (void)bf16;
  const size_t scores = (size_t)tb * score_stride * sizeof(double);
  const size_t sums = (size_t)tb * 4 * 128 * sizeof(double);  // phase 0: [TB][4 waves][D <= 128]
  return scores > sums ? scores : sums;
}

hipError_t launch_route(const RouteArgs& a, bool bf16, int head_dim, int tb, hipStream_t s) {
  const dim3 grid(((a.n_qb + tb - 1) / tb) * a.n_kv_heads);
  const dim3 block(256);
  const size_t lds = route_lds_bytes(tb, a.score_stride, bf16);
#define HGA_ROUTE(T, D, TB) hipLaunchKernelGGL((route_kernel<T, D, TB>), grid, block, lds, s, a)
  if (!bf16) {  // float32 is built for head_dim 64 only
    if (tb == 1) HGA_ROUTE(float, 64, 1); else if (tb == 2) HGA_ROUTE(float, 64, 2); else HGA_ROUTE(float, 64, 4);
  } else if (head_dim == 64) {
    if (tb == 1) HGA_ROUTE(__bf16, 64, 1); else if (tb == 2) HGA_ROUTE(__bf16, 64, 2); else HGA_ROUTE(__bf16, 64, 4);
  } else {
    if (tb == 1) HGA_ROUTE(__bf16, 128, 1); else if (tb == 2) HGA_ROUTE(__bf16, 128, 2); else HGA_ROUTE(__bf16, 128, 4);
  }
#undef HGA_ROUTE
  return hipGetLastError();
}

}  // namespace hga
