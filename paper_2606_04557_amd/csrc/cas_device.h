// Device helpers for the libcas kernels on gfx950 (CDNA4).
//
// Matrix products use the 32x32 MFMA shapes:
//   bf16: v_mfma_f32_32x32x16_bf16  (A, B: 8 bf16 per lane; C: 16 fp32)
//   fp32: v_mfma_f32_32x32x2f32     (A, B: 1 fp32 per lane;  C: 16 fp32)
// Operand layout for lane L = 32*G + n (G = L / 32):
//   A[m][k]: lane (G, m) holds row m, k = G*KH .. G*KH + KH - 1   (KH = K/2)
//   B[k][n]: lane (G, n) holds column n, the same k range
//   C[m][n]: lane (G, n) holds column n, rows crow(j, G) for j = 0..15
// A C fragment therefore holds, per lane, one column and 16 rows; fed back as
// the B operand of a product that reduces over those rows, register j of
// group G must stand for reduction index crow(j, G). "Octet" tiles in LDS
// (below) store the other operand of such a product with its reduction index
// in that same order, so one 16-byte LDS read gives a whole A fragment.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cas_internal.h"

namespace cas {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Row of the 32x32 C fragment held in register j by lane group G.
__device__ __forceinline__ constexpr int crow(int j, int G) {
  return ((j >> 2) << 3) + (G << 2) + (j & 3);
}

template <typename T>
struct Mma;

template <>
struct Mma<__bf16> {
  static constexpr int kStep = 16;   // K per instruction
  using Frag = bf16x8;
  __device__ __forceinline__ static f32x16 run(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static Frag zero() {
    Frag z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
    return z;
  }
};

template <>
struct Mma<float> {
  static constexpr int kStep = 2;
  using Frag = float;
  __device__ __forceinline__ static f32x16 run(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static Frag zero() { return 0.0f; }
};

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

// Row stride (elements) of a row-layout LDS tile: 16 bytes of padding per row
// spread consecutive rows over different banks.
template <typename T, int D>
__device__ __forceinline__ constexpr int lds_row_stride() {
  return D + 16 / (int)sizeof(T);
}

// Operand fragment for a product reducing over the channel axis: row `row`
// of a row-layout tile, channels step*kStep + G*kStep/2 ...
template <typename T, int D>
__device__ __forceinline__ typename Mma<T>::Frag row_frag(const T *tile, int row, int step, int G) {
  constexpr int RS = lds_row_stride<T, D>();
  constexpr int KH = Mma<T>::kStep / 2;
  const T *p = tile + row * RS + step * Mma<T>::kStep + G * KH;
  if constexpr (sizeof(T) == 2) {
    return *reinterpret_cast<const bf16x8 *>(p);
  } else {
    return *p;
  }
}

// The same fragment read straight from global memory.
template <typename T>
__device__ __forceinline__ typename Mma<T>::Frag global_frag(const T *rowp, int step, int G) {
  constexpr int KH = Mma<T>::kStep / 2;
  const T *p = rowp + step * Mma<T>::kStep + G * KH;
  if constexpr (sizeof(T) == 2) {
    return *reinterpret_cast<const bf16x8 *>(p);
  } else {
    return *p;
  }
}

// Octet layout (bf16 only): a tile of R rows (R a multiple of 32) and D
// channels stored as [R/8 octets][D][8]. Octet o = 4*sub + 2*s + G of 32-row
// subtile `sub` holds rows 32*sub + 16*s + 4*G + {0,1,2,3,8,9,10,11}, i.e. the
// rows crow(8s .. 8s+7, G) -- exactly the reduction indices that C-fragment
// registers 8s..8s+7 of group G stand for. Lane (G, m) then reads the A
// fragment A[m = channel][k = those 8 rows] with one 16-byte load.
__device__ __forceinline__ int octet_row(int o, int e) {
  const int sub = o >> 2, s = (o >> 1) & 1, G = o & 1;
  return 32 * sub + 16 * s + 4 * G + (e & 3) + ((e >> 2) << 3);
}

template <int D>
__device__ __forceinline__ bf16x8 octet_frag(const __bf16 *oct, int sub, int s, int G, int ch) {
  const int o = 4 * sub + 2 * s + G;
  return *reinterpret_cast<const bf16x8 *>(oct + ((size_t)o * D + ch) * 8);
}

// Transposed operand fragment for fp32 tiles (row layout): the value of row
// crow(s, G) of subtile `sub` at channel ch (one element per lane per step).
template <int D>
__device__ __forceinline__ float trans_frag_f32(const float *tile, int sub, int s, int G, int ch) {
  constexpr int RS = lds_row_stride<float, D>();
  return tile[(32 * sub + crow(s, G)) * RS + ch];
}

// ---------------------------------------------------------------------------
// Global -> LDS tile loaders. `rowptr(r)` gives the address of row r; rows at
// or beyond `nvalid` are never read and are stored as zeros.
// ---------------------------------------------------------------------------

template <typename T, int D, int R, typename RowPtr>
__device__ __forceinline__ void load_rows(T *tile, RowPtr rowptr, int nvalid, int tid) {
  constexpr int CH = 16 / (int)sizeof(T);     // elements per 16-byte chunk
  constexpr int CPR = D / CH;                 // chunks per row
  constexpr int TOTAL = R * CPR;
  constexpr int RS = lds_row_stride<T, D>();
  static_assert(TOTAL % kThreads == 0, "tile must split evenly over the workgroup");
  u32x4 buf[TOTAL / kThreads];
#pragma unroll
  for (int i = 0; i < TOTAL / kThreads; ++i) {
    const int c = tid + i * kThreads;
    const int r = c / CPR, cc = c % CPR;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < nvalid) v = *reinterpret_cast<const u32x4 *>(rowptr(r) + cc * CH);
    buf[i] = v;
  }
#pragma unroll
  for (int i = 0; i < TOTAL / kThreads; ++i) {
    const int c = tid + i * kThreads;
    const int r = c / CPR, cc = c % CPR;
    *reinterpret_cast<u32x4 *>(tile + r * RS + cc * CH) = buf[i];
  }
}

__device__ __forceinline__ uint32_t lo16(uint32_t w) { return w & 0xffffu; }
__device__ __forceinline__ uint32_t hi16(uint32_t w) { return w >> 16; }

// bf16 tile of R rows into the octet layout, and optionally also into the row
// layout. Each thread moves 8-row x 8-channel blocks and transposes them in
// registers.
template <int D, int R, bool ALSO_ROWS, typename RowPtr>
__device__ __forceinline__ void load_octets(__bf16 *oct, __bf16 *rows_tile, RowPtr rowptr,
                                            int nvalid, int tid) {
  constexpr int NB = (R / 8) * (D / 8);
  constexpr int RS = lds_row_stride<__bf16, D>();
  for (int blk = tid; blk < NB; blk += kThreads) {
    const int o = blk / (D / 8), db = blk % (D / 8);
    u32x4 r[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = octet_row(o, e);
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row < nvalid) v = *reinterpret_cast<const u32x4 *>(rowptr(row) + db * 8);
      r[e] = v;
    }
    if constexpr (ALSO_ROWS) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int row = octet_row(o, e);
        *reinterpret_cast<u32x4 *>(rows_tile + row * RS + db * 8) = r[e];
      }
    }
    // out[c] = (r[0][c], r[1][c], ..., r[7][c]) for channel c = db*8 + 0..7
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int w = c >> 1;
      u32x4 outv;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t a = (c & 1) ? hi16(r[2 * p][w]) : lo16(r[2 * p][w]);
        const uint32_t b = (c & 1) ? hi16(r[2 * p + 1][w]) : lo16(r[2 * p + 1][w]);
        outv[p] = a | (b << 16);
      }
      *reinterpret_cast<u32x4 *>(oct + ((size_t)o * D + db * 8 + c) * 8) = outv;
    }
  }
}

__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32, 64); }

// Stores of 4 consecutive channels.
__device__ __forceinline__ void store4(__bf16 *p, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  v[2] = (__bf16)c;
  v[3] = (__bf16)d;
  *reinterpret_cast<bf16x4 *>(p) = v;
}
__device__ __forceinline__ void store4(float *p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *reinterpret_cast<f32x4 *>(p) = v;
}

template <typename T>
__device__ __forceinline__ float to_f32(T x) {
  return (float)x;
}

}  // namespace cas
