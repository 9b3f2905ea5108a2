// Key summaries (Sec. 2.1 items 1-2, built from the keys attention uses):
// the mean key of every complete g-token group and C-token chunk.
//
// One workgroup per (chunk, kv head); thread (group, column) owns one group
// of g tokens and one 16-byte slice of the head's row and issues its rows'
// loads eight at a time, so a chunk's loads are in flight together and every
// K byte is read once with coalesced 16-byte loads. Group sums are taken in
// float64 in row order and the chunk sum adds the group sums in group order,
// one thread per (column, element); each is rounded once to float32. For
// bf16 keys (8 significant bits) whose magnitudes span less than 2^39 these
// sums are exact, so bit-identical key chunks give bit-identical summaries
// wherever they sit.
#include "hga_device.h"
#include "hga_kernels.h"

namespace hga {

template <typename T>
__global__ __launch_bounds__(1024) void summaries_kernel(SummaryArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int E2 = 16 / EB;  // elements per 16-byte slice
  const int g = 1 << a.group_shift;
  const int n_grp = 64 >> a.group_shift;      // groups per chunk
  const int cols = a.head_dim / E2;           // 16-byte slices per head row
  const int h = blockIdx.x % a.n_kv_heads;
  const int64_t c = a.t_begin / 64 + blockIdx.x / a.n_kv_heads;  // absolute chunk id
  const int64_t t0 = c * 64;
  const int col = threadIdx.x % cols, grp = threadIdx.x / cols;
  const int d0 = col * E2;
  extern __shared__ double s_grp[];           // [group][column][8] group sums
  const int n_tok = (int)min<int64_t>(64, a.t_end - t0);

  double gsum[E2];
#pragma unroll
  for (int e = 0; e < E2; ++e) gsum[e] = 0.0;
  const char* Kb = static_cast<const char*>(a.K) + ((int64_t)h * a.k_head + d0) * EB;
  const int tg = grp * g;
  const int tend = min(tg + g, n_tok);
  // batches of eight rows: all of a batch's loads are issued before the
  // first is summed. Rows past the group's end read row tg again and their
  // sum is discarded by a select, not a branch: a branch lets the compiler
  // sink each load into it, and the eight loads then wait one after another.
  for (int tb = tg; tb < tend; tb += 8) {
    uint4 raw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int tt = tb + i < tend ? tb + i : tg;
      raw[i] = *reinterpret_cast<const uint4*>(Kb + (t0 + tt) * a.k_tok * EB);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the sums after the last load is issued
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool ok = tb + i < tend;
      const uint32_t w[4] = {raw[i].x, raw[i].y, raw[i].z, raw[i].w};
#pragma unroll
      for (int e = 0; e < E2; ++e) {
        float x;
        if constexpr (EB == 2) x = bf16_bits_to_float((w[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
        else x = __uint_as_float(w[e]);
        const double s = gsum[e] + (double)x;
        gsum[e] = ok ? s : gsum[e];
      }
    }
  }
  // the chunk's group sums meet in LDS before any store is issued: a
  // barrier waits for every outstanding memory operation of the wave,
  // stores included
  const bool closed = n_tok == 64;  // the chunk is complete: it has a chunk summary
  if (closed) {
#pragma unroll
    for (int e = 0; e < E2; ++e) s_grp[(grp * cols + col) * 8 + e] = gsum[e];
    __syncthreads();
  }
  if (tg + g <= n_tok) {
    const int64_t j = (t0 + tg) >> a.group_shift;
    const double inv = ldexp(1.0, -a.group_shift);  // 1/g exactly
#pragma unroll
    for (int e = 0; e < E2; e += 4)
      *reinterpret_cast<f32x4*>(a.group_sum + quad_off(h, (d0 + e) / 4, j, a.head_dim, a.group_cap)) =
          f32x4{(float)(gsum[e] * inv), (float)(gsum[e + 1] * inv), (float)(gsum[e + 2] * inv),
                (float)(gsum[e + 3] * inv)};
  }
  if (!closed) return;
  // chunk sum: thread (column, element) adds the chunk's group sums in group
  // order (the same order for every element) and stores its float; the four
  // lanes of a 16-byte quad store together
  const int n_el = cols * E2;  // one more pass when a chunk has fewer than E2 groups
  for (int it = threadIdx.x; it < n_el; it += blockDim.x) {
    const int cc = it % cols, e = it / cols;
    double csum = 0.0;
    for (int q = 0; q < n_grp; ++q) csum += s_grp[(q * cols + cc) * 8 + e];
    const int dd = cc * E2 + e;
    a.chunk_sum[quad_off(h, dd / 4, c, a.head_dim, a.chunk_cap) + dd % 4] = (float)(csum * (1.0 / 64.0));
  }
}

hipError_t launch_summaries(const SummaryArgs& a, bool bf16, hipStream_t s) {
  const int64_t first = a.t_begin / 64;
  const int64_t last = (a.t_end + 63) / 64;
  const int n_chunks = (int)(last - first);
  const int cols = a.head_dim / (bf16 ? 8 : 4);
  const int threads = cols * (64 >> a.group_shift);  // <= 16 * 64
  const dim3 grid(n_chunks * a.n_kv_heads);
  const size_t lds = (size_t)threads * 8 * sizeof(double);
  if (bf16)
    hipLaunchKernelGGL(summaries_kernel<__bf16>, grid, dim3(threads), lds, s, a);
  else
    hipLaunchKernelGGL(summaries_kernel<float>, grid, dim3(threads), lds, s, a);
  return hipGetLastError();
}

}  // namespace hga
