// Key summaries (Sec. 2.1, "two levels of key summaries" from the projected
// keys): the mean key of every complete g-token group and C-token chunk.
//
// One workgroup per chunk; each thread owns one 16-byte column slice of the
// token row (all kv heads side by side) and walks the chunk's 64 tokens, so
// every K byte is read exactly once with fully coalesced 16-byte loads. Sums
// are exact in float64 (bf16 inputs have 8 significant bits) and rounded once
// to float32, which makes bit-identical key chunks give bit-identical
// summaries wherever they sit.
#include "hga_device.h"
#include "hga_kernels.h"

namespace hga {

template <typename T>
__global__ __launch_bounds__(256) void summaries_kernel(SummaryArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E2 = 16 / EB;  // elements per 16-byte slice
  const int C = 64;
  const int g = 1 << a.group_shift;
  const int64_t c = a.t_begin / C + blockIdx.x;  // absolute chunk id
  const int64_t t0 = c * C;
  const int cols = a.n_kv_heads * a.head_dim / E2;
  const char* Kb = static_cast<const char*>(a.K);

  for (int col = threadIdx.x; col < cols; col += blockDim.x) {
    const int hh = (col * E2) / a.head_dim;
    const int d0 = (col * E2) % a.head_dim;
    double gsum[E2], csum[E2];
#pragma unroll
    for (int e = 0; e < E2; ++e) csum[e] = 0.0;
    const int n_tok = (int)min<int64_t>(C, a.t_end - t0);
    for (int tg = 0; tg < n_tok; tg += g) {
#pragma unroll
      for (int e = 0; e < E2; ++e) gsum[e] = 0.0;
      const bool complete = tg + g <= n_tok;
      for (int tt = tg; tt < min(tg + g, n_tok); ++tt) {
        const int64_t off = ((t0 + tt) * a.k_tok + (int64_t)hh * a.k_head + d0) * EB;
        const uint4 raw = *reinterpret_cast<const uint4*>(Kb + off);
        const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
        for (int e = 0; e < E2; ++e) {
          float x;
          if constexpr (EB == 2) {
            x = bf16_bits_to_float((w[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
          } else {
            x = __uint_as_float(w[e]);
          }
          gsum[e] += (double)x;
        }
      }
      if (complete) {
        const int64_t j = (t0 + tg) >> a.group_shift;
        float* dst = a.group_sum + ((int64_t)hh * a.group_cap + j) * a.head_dim + d0;
        const double inv = 1.0 / (double)g;
#pragma unroll
        for (int e = 0; e < E2; e += 4) {
          f32x4 v = {(float)(gsum[e] * inv), (float)(gsum[e + 1] * inv),
                     (float)(gsum[e + 2] * inv), (float)(gsum[e + 3] * inv)};
          *reinterpret_cast<f32x4*>(dst + e) = v;
        }
      }
#pragma unroll
      for (int e = 0; e < E2; ++e) csum[e] += gsum[e];
    }
    if (n_tok == C) {
      float* dst = a.chunk_sum + ((int64_t)hh * a.chunk_cap + c) * a.head_dim + d0;
#pragma unroll
      for (int e = 0; e < E2; e += 4) {
        f32x4 v = {(float)(csum[e] / C), (float)(csum[e + 1] / C), (float)(csum[e + 2] / C),
                   (float)(csum[e + 3] / C)};
        *reinterpret_cast<f32x4*>(dst + e) = v;
      }
    }
  }
}

hipError_t launch_summaries(const SummaryArgs& a, bool bf16, hipStream_t s) {
  const int64_t first = a.t_begin / 64;
  const int64_t last = (a.t_end + 63) / 64;
  const int n_chunks = (int)(last - first);
  const int cols = a.n_kv_heads * a.head_dim / (bf16 ? 8 : 4);
  const int threads = cols >= 256 ? 256 : ((cols + 63) / 64) * 64;
  if (bf16)
    hipLaunchKernelGGL(summaries_kernel<__bf16>, dim3(n_chunks), dim3(threads), 0, s, a);
  else
    hipLaunchKernelGGL(summaries_kernel<float>, dim3(n_chunks), dim3(threads), 0, s, a);
  return hipGetLastError();
}

}  // namespace hga
