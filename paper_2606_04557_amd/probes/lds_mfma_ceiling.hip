// What rate can a bf16 MFMA stream sustain on gfx950 when every
// v_mfma_f32_32x32x16_bf16 takes one 1 KiB operand fragment from LDS, the
// pattern of the attention kernels (one operand stationary in registers, the
// other streamed through LDS)? Each variant runs one 512-thread workgroup
// (8 waves, two per SIMD) per compute unit for a fixed number of steps on
// random bf16 data (magnitudes in [1, 2), random signs) and reports TFLOP/s
// from HIP events around the launch. LDS holds 64 KiB of such data and is
// never written in the timed loop; every LDS read stays inside it.
//
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       lds_mfma_ceiling.hip -o lds_mfma_ceiling && ./lds_mfma_ceiling
//
// Variants (a "phase" is 32 MFMAs of one wave):
//   reg        both waves of each SIMD stream MFMAs on register operands
//   lds1       both waves stream MFMAs, each with one LDS fragment
//   lds2       both waves stream MFMAs, one LDS fragment per two MFMAs
//   ldsonly    LDS fragment reads alone (bytes per clock of the LDS)
//   pp_reg     ping-pong: per phase one wave of each SIMD runs 32 MFMAs on
//              register operands while the other converts 32 scores (fma,
//              exp2, bf16 pack); a workgroup barrier ends each phase
//   pp_lds     the same with one LDS fragment per MFMA (the kernels' shape)
//   pp_noexp   pp_lds without the exp2 in the conversion phase
//   pp_sink    pp_lds's loads and waits, but the MFMAs take register operands
//   pp_pre     pp_lds with the first fragments of a matrix phase loaded
//              before the barrier that starts it
//   inter      no barriers: every wave interleaves its own conversion of last
//              step's scores with this step's 32 LDS-fed MFMAs
//   one_blk    one wave per SIMD (4-wave workgroups, the whole register
//              file): 32 MFMAs per step on 16 LDS fragments, each used for
//              two MFMAs, with last step's conversion interleaved
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);  \
      return 1;                                                               \
    }                                                                         \
  } while (0)

namespace {

constexpr int kLds = 64 * 1024;
constexpr int kLead = 6;   // fragments in flight ahead of their MFMA

enum Mode { REG, LDS1, LDS2, LDSONLY, PP_REG, PP_LDS, PP_NOEXP, PP_SINK, PP_PRE, INTER, ONE_BLK };

__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}
// Two bf16 values with magnitude in [1, 2) and random signs.
__device__ __forceinline__ uint32_t two_bf16(uint32_t h) {
  const uint32_t lo = 0x3F80u | (h & 0x7Fu) | (((h >> 7) & 1u) << 15);
  const uint32_t hi = 0x3F80u | ((h >> 8) & 0x7Fu) | (((h >> 15) & 1u) << 15);
  return lo | (hi << 16);
}
__device__ __forceinline__ bf16x8 rand_frag(uint32_t seed) {
  u32x4 u;
#pragma unroll
  for (int i = 0; i < 4; ++i) u[i] = two_bf16(mix(seed * 4 + i));
  return __builtin_bit_cast(bf16x8, u);
}
__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int e = 0; e < 16; ++e) z[e] = 0.f;
  return z;
}
__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 lds_frag(const char *p) { return *reinterpret_cast<const bf16x8 *>(p); }

template <int M>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void probe(int steps, float *out) {
  __shared__ __attribute__((aligned(1024))) char smem[kLds];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < kLds / 4; i += 512) reinterpret_cast<uint32_t *>(smem)[i] = two_bf16(mix(i + blockIdx.x * 77777u));
  __syncthreads();

  bf16x8 kv[8], pk[4];
#pragma unroll
  for (int s = 0; s < 8; ++s) kv[s] = rand_frag(tid * 16 + s + blockIdx.x * 4096);
#pragma unroll
  for (int s = 0; s < 4; ++s) pk[s] = rand_frag(tid * 16 + s + 8 + blockIdx.x * 4096);
  f32x16 acc[4], sp[2];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = zero16();
  sp[0] = zero16();
  sp[1] = zero16();
  // 32 fragments of 1 KiB per window; the waves of each half of the
  // workgroup read one window, as they read a shared operand block.
  const bool grp_a = wave < 4;
  const char *base = smem + (M >= PP_REG && M <= PP_PRE ? (grp_a ? 0 : 32768) : (wave & 1) * 32768) + lane * 16;
  const float c = 0.0883883f, sub = 3.0f;
  u32x4 sink = {0, 0, 0, 0};

  // 32 MFMAs of one wave: 16 score-like (fragment x kv into sp), 16
  // product-like (fragment x packed values into acc).
  bf16x8 pre[kLead];
  auto matrix = [&]() __attribute__((always_inline)) {
    sp[0] = zero16();
    sp[1] = zero16();
    bf16x8 ring[kLead + 1];
    if constexpr (M == PP_PRE) {
#pragma unroll
      for (int k = 0; k < kLead; ++k) ring[k] = pre[k];
    } else if constexpr (M != PP_REG) {
#pragma unroll
      for (int k = 0; k < kLead; ++k) ring[k] = lds_frag(base + k * 1024);
    }
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 f;
      if constexpr (M == PP_REG) {
        f = kv[(k + 3 + (k >> 3)) & 7];
      } else if constexpr (M == PP_SINK) {
        if (k + kLead < 32)
          ring[(k + kLead) % (kLead + 1)] =
              *(const volatile __attribute__((address_space(3))) bf16x8 *)(base + (k + kLead) * 1024);
        asm volatile("" ::"v"(ring[k % (kLead + 1)]));
        f = kv[(k + 3 + (k >> 3)) & 7];
      } else {
        if (k + kLead < 32) ring[(k + kLead) % (kLead + 1)] = lds_frag(base + (k + kLead) * 1024);
        f = ring[k % (kLead + 1)];
      }
      if (k < 16) sp[k >> 3] = mfma(f, kv[k & 7], sp[k >> 3]);
      else acc[(k - 16) >> 2] = mfma(f, pk[k & 3], acc[(k - 16) >> 2]);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Conversion of the scores: fma, exp2, bf16 pack (32 values per lane).
  auto convert = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float v = fmaf(sp[j][e], c, -sub);
        if constexpr (M != PP_NOEXP) v = __builtin_amdgcn_exp2f(v);
        sp[j][e] = v;
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (__bf16)sp[j][8 * h + e];
        pk[2 * j + h] = o;
      }
    }
  };
  auto preload = [&]() __attribute__((always_inline)) {
    if constexpr (M == PP_PRE) {
#pragma unroll
      for (int k = 0; k < kLead; ++k) pre[k] = lds_frag(base + k * 1024);
    }
  };
  auto barrier = [&]() __attribute__((always_inline)) {
    if constexpr (M != PP_PRE) __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  if constexpr (M == REG || M == LDS1 || M == LDS2 || M == LDSONLY) {
    bf16x8 a[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) a[s] = rand_frag(tid * 16 + s + 8 + blockIdx.x * 4096);
    for (int it = 0; it < steps; ++it) {
      if constexpr (M == REG) {
#pragma unroll
        for (int k = 0; k < 32; ++k) acc[k & 3] = mfma(a[k & 7], kv[(k >> 2) & 7], acc[k & 3]);
      } else if constexpr (M == LDS1) {
        bf16x8 ring[kLead + 1];
#pragma unroll
        for (int k = 0; k < kLead; ++k) ring[k] = lds_frag(base + k * 1024);
#pragma unroll
        for (int k = 0; k < 32; ++k) {
          if (k + kLead < 32) ring[(k + kLead) % (kLead + 1)] = lds_frag(base + (k + kLead) * 1024);
          acc[k & 3] = mfma(ring[k % (kLead + 1)], kv[(k >> 2) & 7], acc[k & 3]);
        }
      } else if constexpr (M == LDS2) {
        bf16x8 ring[kLead + 1];
#pragma unroll
        for (int k = 0; k < kLead; ++k) ring[k] = lds_frag(base + k * 1024);
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          if (k + kLead < 16) ring[(k + kLead) % (kLead + 1)] = lds_frag(base + (k + kLead) * 1024);
          acc[(2 * k) & 3] = mfma(ring[k % (kLead + 1)], kv[k & 7], acc[(2 * k) & 3]);
          acc[(2 * k + 1) & 3] = mfma(ring[k % (kLead + 1)], a[k & 7], acc[(2 * k + 1) & 3]);
        }
      } else {
#pragma unroll
        for (int k = 0; k < 32; ++k) sink ^= *reinterpret_cast<const u32x4 *>(base + k * 1024);
      }
      asm volatile("" ::: "memory");
    }
  } else if constexpr (M == INTER) {
    f32x16 sq[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) sq[j][e] = 0.01f * e;
    for (int it = 0; it < steps; ++it) {
      bf16x8 ring[kLead + 1];
#pragma unroll
      for (int k = 0; k < kLead; ++k) ring[k] = lds_frag(base + k * 1024);
      f32x16 sn[2] = {zero16(), zero16()};
      bf16x8 pn[4];
#pragma unroll
      for (int k = 0; k < 32; ++k) {
        if (k + kLead < 32) ring[(k + kLead) % (kLead + 1)] = lds_frag(base + (k + kLead) * 1024);
        if (k < 16) sn[k >> 3] = mfma(ring[k % (kLead + 1)], kv[k & 7], sn[k >> 3]);
        else acc[(k - 16) >> 2] = mfma(ring[k % (kLead + 1)], pk[k & 3], acc[(k - 16) >> 2]);
        const int j = k >> 4, e = k & 15;   // one score of last step per MFMA
        sq[j][e] = __builtin_amdgcn_exp2f(fmaf(sq[j][e], c, -sub));
        if ((k & 7) == 7) {
          const int h = (k >> 3) & 1;
          bf16x8 o;
#pragma unroll
          for (int q = 0; q < 8; ++q) o[q] = (__bf16)sq[j][8 * h + q];
          pn[2 * j + h] = o;
        }
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) pk[s] = pn[s];
      sq[0] = sn[0];
      sq[1] = sn[1];
      asm volatile("" ::: "memory");
    }
  } else {
    if (grp_a) preload();
    for (int it = 0; it < steps; ++it) {
      if (grp_a) matrix();
      else {
        convert();
        preload();
      }
      barrier();
      if (grp_a) {
        convert();
        preload();
      } else {
        matrix();
      }
      barrier();
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  s += (float)(sink[0] ^ sink[1] ^ sink[2] ^ sink[3]) * 1e-30f;
  out[blockIdx.x * 512 + tid] = s;
}

// One wave per SIMD: each LDS fragment feeds two MFMAs (two stationary
// operand sets), and the conversion of last step's 32 scores per lane is
// interleaved with this step's 32 MFMAs.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void probe_one(int steps, float *out) {
  __shared__ __attribute__((aligned(1024))) char smem[kLds];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int i = tid; i < kLds / 4; i += 256) reinterpret_cast<uint32_t *>(smem)[i] = two_bf16(mix(i + blockIdx.x * 77777u));
  __syncthreads();
  bf16x8 k0[8], k1[8], pk[4];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    k0[s] = rand_frag(tid * 32 + s + blockIdx.x * 8192);
    k1[s] = rand_frag(tid * 32 + s + 8 + blockIdx.x * 8192);
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) pk[s] = rand_frag(tid * 32 + s + 16 + blockIdx.x * 8192);
  f32x16 acc[4], sq[2];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = zero16();
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) sq[j][e] = 0.01f * e;
  const char *base = smem + lane * 16;
  const float c = 0.0883883f, sub = 3.0f;
  for (int it = 0; it < steps; ++it) {
    bf16x8 ring[kLead + 1];
#pragma unroll
    for (int k = 0; k < kLead; ++k) ring[k] = lds_frag(base + k * 1024);
    f32x16 sn[2] = {zero16(), zero16()};
    bf16x8 pn[4];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      if (k + kLead < 16) ring[(k + kLead) % (kLead + 1)] = lds_frag(base + (k + kLead) * 1024);
      const bf16x8 f = ring[k % (kLead + 1)];
      if (k < 8) {   // scores of two key halves from one fragment
        sn[0] = mfma(f, k0[k & 7], sn[0]);
        sn[1] = mfma(f, k1[k & 7], sn[1]);
      } else {       // products of two channel halves from one fragment
        acc[(k - 8) >> 2] = mfma(f, pk[k & 3], acc[(k - 8) >> 2]);
        acc[2 + ((k - 8) >> 2)] = mfma(f, pk[(k + 1) & 3], acc[2 + ((k - 8) >> 2)]);
      }
      // two scores of last step per fragment
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int q = 2 * k + t, j = q >> 4, e = q & 15;
        sq[j][e] = __builtin_amdgcn_exp2f(fmaf(sq[j][e], c, -sub));
      }
      if ((k & 3) == 3) {
        const int q = 2 * k + 1, j = q >> 4, h = (q >> 3) & 1;
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (__bf16)sq[j][8 * h + e];
        pn[2 * j + h] = o;
      }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) pk[s] = pn[s];
    sq[0] = sn[0];
    sq[1] = sn[1];
    asm volatile("" ::: "memory");
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  out[blockIdx.x * 512 + tid] = s;
}

// Runs variant M over `steps` steps; MFMAs (or 1 KiB LDS reads) per wave and step.
template <int M>
int run(const char *name, int steps, int mfma_per_wave_step, int lds_kib_per_wave_step, int cus, float *out) {
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  if constexpr (M == ONE_BLK) probe_one<<<cus, 256>>>(steps / 10, out);   // warm-up
  else probe<M><<<cus, 512>>>(steps / 10, out);
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  CHECK(hipEventRecord(e0));
  if constexpr (M == ONE_BLK) probe_one<<<cus, 256>>>(steps, out);
  else probe<M><<<cus, 512>>>(steps, out);
  CHECK(hipGetLastError());
  CHECK(hipEventRecord(e1));
  CHECK(hipEventSynchronize(e1));
  float ms = 0.f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  const double waves = cus * (M == ONE_BLK ? 4.0 : 8.0);
  const double tflops = waves * steps * mfma_per_wave_step * 32768.0 / (ms * 1e-3) / 1e12;
  const double lds_tbs = waves * steps * lds_kib_per_wave_step * 1024.0 / (ms * 1e-3) / 1e12;
  printf("%-10s %9.3f ms  %8.1f TFLOP/s  LDS reads %6.1f TB/s (%.0f B per CU per ns)\n", name, ms, tflops, lds_tbs,
         lds_tbs * 1e12 / cus / 1e9);
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  return 0;
}

}  // namespace

int main() {
  hipDeviceProp_t prop;
  CHECK(hipGetDeviceProperties(&prop, 0));
  const int cus = prop.multiProcessorCount;
  printf("%s: %d compute units, one 8-wave workgroup each\n", prop.gcnArchName, cus);
  float *out = nullptr;
  CHECK(hipMalloc(&out, (size_t)cus * 512 * sizeof(float)));
  const int n = 40000;   // steps of 32 MFMAs per wave (ping-pong: n/2 steps of two phases)
  int rc = 0;
  rc |= run<REG>("reg", n, 32, 0, cus, out);
  rc |= run<LDS1>("lds1", n, 32, 32, cus, out);
  rc |= run<LDS2>("lds2", n, 32, 16, cus, out);
  rc |= run<LDSONLY>("ldsonly", 4 * n, 0, 32, cus, out);
  rc |= run<PP_REG>("pp_reg", n / 2, 32, 0, cus, out);
  rc |= run<PP_LDS>("pp_lds", n / 2, 32, 32, cus, out);
  rc |= run<PP_NOEXP>("pp_noexp", n / 2, 32, 32, cus, out);
  rc |= run<PP_SINK>("pp_sink", n / 2, 32, 32, cus, out);
  rc |= run<PP_PRE>("pp_pre", n / 2, 32, 32, cus, out);
  rc |= run<INTER>("inter", n, 32, 32, cus, out);
  rc |= run<ONE_BLK>("one_blk", n, 32, 16, cus, out);
  rc |= run<REG>("reg", n, 32, 0, cus, out);
  CHECK(hipFree(out));
  return rc;
}
