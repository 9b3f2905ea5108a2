// Device-side building blocks of the gfx950 HGA kernels: element traits,
// MFMA wrappers, bf16 conversion and the LDS tile layouts that feed the
// 32x32 matrix-core instructions.
//
// MFMA lane layout used throughout (32x32xK, wave64, lane l, half hh = l/32):
//   A operand : row m = l%32,     k = E*hh + j   (j < E elements per lane)
//   B operand : col n = l%32,     k = E*hh + j
//   C/D       : col n = l%32,     row m = 8*(v/4) + 4*hh + v%4 (v < 16)
// A C/D tile therefore serves directly as a B operand of the next product
// (its column index stays the column), provided the k order of the next
// product follows the row order of the C tile. `kpos_of` gives that order.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hga {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <typename T> struct Elem;

// bf16 storage (uint16 bit patterns in memory), 32x32x16 bf16 MFMA.
template <> struct Elem<__bf16> {
  static constexpr int kBytes = 2;
  static constexpr int E = 8;       // elements per lane per MFMA operand
  static constexpr int KSTEP = 16;  // k covered by one MFMA
  using Frag = bf16x8;
  __device__ static inline f32x16 mma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline Frag load_frag(const char* p) { return *reinterpret_cast<const Frag*>(p); }
  __device__ static inline Frag frag_from(const float* x) {
    Frag f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = (__bf16)x[j];
    return f;
  }
};

// fp32 storage, 32x32x2 f32 MFMA (full fp32 products).
template <> struct Elem<float> {
  static constexpr int kBytes = 4;
  static constexpr int E = 1;
  static constexpr int KSTEP = 2;
  using Frag = float;
  __device__ static inline f32x16 mma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline Frag load_frag(const char* p) { return *reinterpret_cast<const float*>(p); }
  __device__ static inline Frag frag_from(const float* x) { return x[0]; }
};

__device__ inline float bf16_bits_to_float(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// Row `tok` of a tensor whose rows are `stride_bytes` apart: the ABI keeps
// positions below 2^31 and strides below 4 GB, so the offset is one 32 x 32 ->
// 64-bit multiply-add.
__device__ inline const char* row_ptr(const char* base, int64_t tok, int64_t stride_bytes) {
  return base + (uint64_t)(uint32_t)tok * (uint32_t)stride_bytes;
}

// Round-to-nearest-even float -> bf16 bit pattern (finite inputs).
__device__ inline uint32_t float_to_bf16_bits(float f) {
  __bf16 b = (__bf16)f;
  return (uint32_t)__builtin_bit_cast(uint16_t, b);
}

// Position, inside the k axis of a 64-wide product, of key (or query) `r`
// (0..63) of a tile whose scores were produced as two 32x32 C tiles.
// For MFMA k-step s, half hh and element j the product consumes C row
// m = 8*(v/4) + 4*hh + v%4 of tile t, with v = E*(s % (16/E)) + j; its
// position on the k axis is KSTEP*s + E*hh + j. This is the inverse map.
template <int E>
__device__ __host__ constexpr int kpos_of(int r) {
  const int t = r >> 5, m = r & 31;
  const int hh = (m >> 2) & 1;
  const int v = 4 * (m >> 3) + (m & 3);
  constexpr int VPS = 16 / E;  // k-steps per 32-row C tile
  const int s = t * VPS + v / E;
  const int j = v % E;
  return 2 * E * s + E * hh + j;
}

// ---------------------------------------------------------------------------
// LDS tile layouts (one 64-token tile of one head, head dim D).
//
// Row tile [64][D]: token r is stored in physical row pi(r), each row padded
// by 16 bytes, where pi(r) = (r & ~15) | ((r & 3) << 2) | ((r >> 2) & 3)
// swaps the two 2-bit fields of the row index inside each group of 16. The
// two ways the kernels read the tile then hit distinct LDS banks per pass:
//  - an MFMA operand load (16 lanes = 16 consecutive tokens, one 16-byte
//    piece each): pi permutes each group of 16 rows, and padded rows start
//    4 banks apart, so the 16 pieces cover all 64 banks;
//  - a transpose load (32 lanes = 4 tokens starting at a multiple of 4,
//    times 64 contiguous bytes): pi puts the 4 tokens 4 rows = 16 banks
//    apart, so the four 16-bank windows are disjoint.
// pi keeps bits >= 4, so offsets of tokens 16 apart stay immediate.
// Transposed tile [D][64] (fp32 only): element (d, kpos) holds the token
// whose k position is kpos; rows padded to 65 words.
// ---------------------------------------------------------------------------
template <typename T, int D>
struct Tile {
  static constexpr int kRowPitch = D * Elem<T>::kBytes + 16;
  static constexpr int kRowBytes = 64 * kRowPitch;
  static constexpr int kTPitch = Elem<T>::kBytes == 2 ? 128 : 65 * 4;
  static constexpr int kTBytes = D * kTPitch;

  __device__ static inline int row_perm(int r) { return (r & ~15) | ((r & 3) << 2) | ((r >> 2) & 3); }

  // Byte offset of element d of token row r.
  __device__ static inline int row_off(int r, int d) { return row_perm(r) * kRowPitch + d * Elem<T>::kBytes; }

  __device__ static inline int swz(int d) { return ((d >> 1) ^ (d >> 3)) & 7; }

  // Byte offset of element (d, kpos) of a transposed tile.
  __device__ static inline int t_off(int d, int kpos) {
    if constexpr (Elem<T>::kBytes == 2) {
      return d * 128 + (((kpos >> 3) ^ swz(d)) << 4) + ((kpos & 7) << 1);
    } else {
      return (d * 65 + kpos) * 4;
    }
  }
};

// Operand fragment whose lane index runs along the columns of a row-major
// bf16 LDS tile, read with the gfx950 LDS transpose load (ds_read_b64_tr_b16).
// Within each 16-lane group, source lane i points at row r + i/4, columns
// 4*(i%4)..+3; lane j then receives column j of rows r..r+3. The fragment of
// lane l is column col_base + l%32 of rows ra..ra+3 (elements 0-3) and
// rb..rb+3 (elements 4-7), ra and rb chosen by the caller for its lane half.
typedef short s16x4 __attribute__((ext_vector_type(4)));
template <typename TL>
__device__ inline bf16x8 tr_frag(const char* tile, int col_base, int ra, int rb, int lane) {
  const int i = lane & 15;
  const int col = col_base + 16 * ((lane >> 4) & 1) + 4 * (i & 3);
  typedef __attribute__((address_space(3))) s16x4* lds_s4;
  const s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(tile + TL::row_off(ra + (i >> 2), col)));
  const s16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(tile + TL::row_off(rb + (i >> 2), col)));
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 both = __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, both);
}

// Wave-wide helpers.
__device__ inline float xor32(float x) { return __shfl_xor(x, 32, 64); }

// Barrier of the whole workgroup.
struct WgSync {
  __device__ inline void operator()() { __syncthreads(); }
};

// Barrier of a team of `waves` waves inside a workgroup whose other waves
// run other code (s_barrier would wait for them too). Each wave adds one to
// an LDS counter (zero before the team's first barrier) and waits until the
// counter reaches `waves` times its own barrier count; release and acquire
// fences at workgroup scope order the team's LDS traffic around it. Every
// wave of the team must call it the same number of times, and the waves of
// a workgroup are resident together, so the wait always ends.
struct WaveGroupSync {
  int* ctr;
  int waves;
  int gen = 0;
  __device__ inline void operator()() {
    ++gen;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    const int target = gen * waves;
    while (__builtin_amdgcn_readfirstlane(__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) <
           target)
      __builtin_amdgcn_s_sleep(1);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
};

// One-way hand-over between teams: the producing wave publishes after its LDS
// writes; a consumer that sees the flag set may read them.
__device__ inline void publish_flag(int* flag) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  if ((threadIdx.x & 63) == 0) __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ inline bool flag_set(int* flag) {
  const int f = __builtin_amdgcn_readfirstlane(__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
  if (f != 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  return f != 0;
}

}  // namespace hga
