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

namespace cas {

// ---------------------------------------------------------------------------
// Swizzled bf16 row tiles for the gfx950 fast path.
//
// A tile of R rows x D bf16 columns is stored with no padding; row r's
// 16-byte chunk c sits at chunk position c ^ swz(r). For D = 128 the swizzle
// swz(r) = 4*(r%4) + (r/4)%4 makes both access patterns conflict-free:
//   * row fragments (lane m reads row m, one chunk): 16 consecutive rows hit
//     16 different bank groups;
//   * transposed fragments (ds_read_b64_tr_b16, 8 rows x 64 bytes): each
//     group of 4 rows covers all 16 bank groups.
// Tiles are filled with direct buffer->LDS copies (buffer_load_dwordx4 ... lds),
// so a wave's 64 lanes write 1 KiB in lane order and the swizzle is applied
// on the global side (lane at chunk position p of row r loads chunk p^swz(r)).
// ---------------------------------------------------------------------------

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;

template <int D>
__device__ __forceinline__ constexpr int swz(int r) {
  if constexpr (D == 128) {
    return ((r & 3) << 2) | ((r >> 2) & 3);
  } else {
    return (r >> 1) & 7;
  }
}

template <int D>
__device__ __forceinline__ int swz_off(int r, int c) {
  return r * (D * 2) + ((c ^ swz<D>(r)) << 4);
}

// Buffer resource over `bytes` bytes from base (raw addressing, no stride);
// loads at offsets beyond it return zero. Direct buffer->LDS copies of 16
// bytes per lane: a wave writes 1 KiB in lane order at lds. Unlike the FLAT
// form, a MUBUF LDS load is tracked on vmcnt alone, so LDS reads issued while
// copies are in flight keep exact lgkmcnt waits.
typedef __amdgpu_buffer_rsrc_t BufRsrc;

__device__ __forceinline__ BufRsrc make_rsrc(const void *base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, 0x00020000);
}

__device__ __forceinline__ void dma16(BufRsrc rs, int byte_off, char *lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t *)lds, 16, byte_off, 0, 0, 0);
}

// Asynchronous copy of R rows into a swizzled tile, shared by NW waves: row r
// starts rowoff(r) elements after base (rowoff increases by at least D per
// row and stays in 32 bits). The buffer resource ends after row nvalid-1
// (>= 1), so rows at or beyond nvalid read as zero. Completion: s_waitcnt
// vmcnt + barrier.
template <int D, int R, int NW, typename RowOff>
__device__ __forceinline__ void dma_tile(char *tile, const __bf16 *base, RowOff rowoff, int nvalid, int wave,
                                         int lane) {
  constexpr int CPR = D / 8;
  constexpr int NI = R * CPR / 64;   // 1 KiB wave instructions per tile
  const BufRsrc rs = make_rsrc(base, (rowoff(nvalid - 1) + D) * 2);
  for (int inst = wave; inst < NI; inst += NW) {
    const int pos = inst * 64 + lane;
    const int r = pos / CPR;
    const int c = (pos % CPR) ^ swz<D>(r);
    dma16(rs, (rowoff(r) + c * 8) * 2, tile + inst * 1024);
  }
}

// Asynchronous copy of 64 consecutive floats (one wave instruction); lanes at
// or beyond n read zero.
__device__ __forceinline__ void dma_f32x64_zero(float *dst, const float *src, int n, int lane) {
  const BufRsrc rs = make_rsrc(src, n * 4);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t *)dst, 4, lane * 4, 0, 0, 0);
}

// Per-lane byte offsets into swizzled tiles. swz(r) is unchanged when r moves
// by a multiple of 16, so fragments of rows r + 16k are the same offsets plus
// a constant: each lane keeps D/16 row-fragment and D/16 transposed-fragment
// offsets and every tile/subtile/buffer is reached by an immediate offset.
//
// Row fragment: lane (G, m) reads row m, chunk 2*st + G (channels 16st+8G..).
template <int D>
struct RowOffsets {
  int off[D / 16];
  __device__ __forceinline__ void init(int m, int G) {
#pragma unroll
    for (int st = 0; st < D / 16; ++st) off[st] = m * (D * 2) + (((2 * st + G) ^ swz<D>(m)) << 4);
  }
};

// Transposed A fragment of a 32x32x16 MFMA from a row tile: lane (G, m)
// receives column dt*32 + m of rows row0 + 4G + {0..3} (slots 0..3) and
// row0 + 8 + 4G + {0..3} (slots 4..7) -- the reduction indices that C
// registers 8s..8s+7 of group G stand for when row0 = 32*sub + 16*s.
// ds_read_b64_tr_b16: within each 16-lane block, output lane 4a+c receives
// element c of the 8 bytes addressed by source lanes a, a+4, a+8, a+12; so
// source lane 16b + j addresses row row0 + 8h + 4(b/2) + j/4 at columns
// dt*32 + 16(b%2) + 4(j%4) .. +3.
template <int D>
struct TrOffsets {
  int off[D / 32][2];
  __device__ __forceinline__ void init(int lane) {
    const int b = lane >> 4, j = lane & 15;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row = 8 * h + 4 * (b >> 1) + (j >> 2);
        const int col = dt * 32 + 16 * (b & 1) + 4 * (j & 3);
        off[dt][h] = row * (D * 2) + (((col >> 3) ^ swz<D>(row)) << 4) + ((col >> 2) & 1) * 8;
      }
  }
};

template <int D>
__device__ __forceinline__ bf16x8 row_frag_at(const char *tile, const RowOffsets<D> &ro, int row0, int st) {
  return *reinterpret_cast<const bf16x8 *>(tile + row0 * (D * 2) + ro.off[st]);
}

template <int D>
__device__ __forceinline__ bf16x8 tr_frag_at(const char *tile, const TrOffsets<D> &to, int row0, int dt) {
  const char *base = tile + row0 * (D * 2);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(base + to.off[dt][0]));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(base + to.off[dt][1]));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  const i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 pack_bf16x8(const f32x16 &x, int s) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)x[8 * s + e];
  return r;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }


__device__ __forceinline__ bool wave_any(bool p) { return __ballot(p) != 0; }

// s_waitcnt for "at most n vector-memory operations of this wave outstanding",
// leaving the export and LDS/scalar counters alone (gfx9 encoding: vmcnt in
// bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8). Direct global->LDS copies
// complete in issue order, so this waits for all but the newest n copies.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Launch tables (segment descriptors, use lists) are written before a kernel
// starts and never during it; reading them through the constant address space
// lets uniform reads become scalar loads.
template <typename T>
__device__ __forceinline__ T load_const(const T *base, int i) {
  static_assert(sizeof(T) % 4 == 0, "4-byte words");
  typedef const __attribute__((address_space(4))) uint32_t cword_t;
  cword_t *w = (cword_t *)(base + i);
  T r;
  uint32_t *rw = reinterpret_cast<uint32_t *>(&r);
#pragma unroll
  for (int k = 0; k < (int)(sizeof(T) / 4); ++k) rw[k] = w[k];
  return r;
}

}  // namespace cas
