// What HBM read rate can the paged decode's access pattern reach on this
// chip? The decode streams, per (request, KV head), key rows of 256 bytes
// (128 bf16 channels) that lie 2 KiB apart (eight KV heads per token) inside
// 16-token pages, the pages named by a page table: four retrieved 1,024-token
// cartridges from a pool of 256, then the request's own 65 tokens. This probe
// reads exactly those bytes of K and V, for 64 requests and 8 KV heads, with
// no arithmetic beyond an XOR fold, and compares it with one sequential
// stream over the whole pool. Each variant is timed with HIP events around
// the launch; a store that the data never triggers keeps the loads alive.
//
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       hbm_read_ceiling.hip -o hbm_read_ceiling && ./hbm_read_ceiling
//
// Variants:
//   seq           grid-stride read of both pools in order (16-byte loads,
//                 U loads in flight per lane)
//   pages U S     the decode's bytes: one 256-thread workgroup per
//                 (request, KV head, key range), S ranges per (request, KV
//                 head), U 32-key tiles of K and V in flight per lane
//   wave S        register loads as in `pages` U 1, but each of the four
//                 waves on every fourth tile of its own (one 16 KiB tile of
//                 K and V per wave and iteration)
//   dma S         the same bytes by direct buffer->LDS copies, each of the
//                 four waves on every fourth tile (the decode kernel's
//                 assignment), one 16 KiB tile (K and V) in flight per wave,
//                 two workgroups per compute unit
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <vector>

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);  \
      return 1;                                                               \
    }                                                                         \
  } while (0)

namespace {

constexpr int kPage = 16;                 // tokens per page
constexpr int kHkv = 8;
constexpr int kD = 128;
constexpr int kCarts = 256, kCartPages = 64;
constexpr int kReqs = 64, kSel = 4, kOwn = 65;
constexpr int kOwnPages = (kOwn + kPage - 1) / kPage;
constexpr int kReqPages = kSel * kCartPages + kOwnPages;       // 261
constexpr int kKvLen = kSel * kCartPages * kPage + kOwn;       // 4,161 keys
constexpr int kTile = 32;
constexpr int kTiles = (kKvLen + kTile - 1) / kTile;          // 131
constexpr int64_t kPages = (int64_t)kCarts * kCartPages + (int64_t)kReqs * kOwnPages;
constexpr int64_t kPoolElems = kPages * kPage * kHkv * kD;     // bf16 elements per pool

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void keep(u32x4 acc, u32x4 *sink) {
  if (acc[0] == 0x9E3779B9u && acc[1] == 0x7F4A7C15u && acc[2] == 0x85EBCA6Bu && acc[3] == 0xC2B2AE35u)
    sink[blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

template <int U>
__global__ __launch_bounds__(256) void seq_kernel(const u32x4 *a, int64_t n, u32x4 *sink) {
  u32x4 acc = {0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + (U - 1) * stride < n; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(a + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
  }
  for (; i < n; i += stride) acc ^= a[i];
  keep(acc, sink);
}

// Lane l of a tile reads 16 bytes (channel chunk l % 16) of keys l / 16 and
// l / 16 + 16; a wave covers four whole 256-byte key rows per load.
template <int U>
__global__ __launch_bounds__(256) void pages_kernel(const uint16_t *kp, const uint16_t *vp, const int *table,
                                                    int splits, u32x4 *sink) {
  const int w = blockIdx.x;
  const int split = w % splits, pair = w / splits;
  const int h = pair % kHkv, r = pair / kHkv;
  const int t0 = (int)((int64_t)kTiles * split / splits), t1 = (int)((int64_t)kTiles * (split + 1) / splits);
  const int *pt = table + r * kReqPages;
  const int c = threadIdx.x & 15, k = threadIdx.x >> 4;   // chunk, key within the half tile
  u32x4 acc = {0, 0, 0, 0};
  for (int t = t0; t < t1; t += U) {
    u32x4 v[U][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tt = t + u;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int key = tt * kTile + half * 16 + k;       // page tt * 2 + half, token k
        if (tt < t1 && key < kKvLen) {
          const int page = pt[tt * 2 + half];
          const int64_t off = (((int64_t)page * kPage + k) * kHkv + h) * kD + c * 8;
          v[u][2 * half] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(kp + off));
          v[u][2 * half + 1] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(vp + off));
        } else {
          v[u][2 * half] = u32x4{0, 0, 0, 0};
          v[u][2 * half + 1] = u32x4{0, 0, 0, 0};
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc ^= v[u][e];
  }
  keep(acc, sink);
}

// Wave w of a workgroup reads tiles t0 + w, t0 + w + 4, ... of its (request,
// KV head): per tile each lane loads 8 pieces of 16 bytes (K and V of keys
// 4 i + lane / 16, chunk lane % 16, i = 0..3), then folds them.
__global__ __launch_bounds__(256) void wave_kernel(const uint16_t *kp, const uint16_t *vp, const int *table,
                                                   int splits, u32x4 *sink) {
  const int w = blockIdx.x;
  const int split = w % splits, pair = w / splits;
  const int h = pair % kHkv, r = pair / kHkv;
  const int t0 = (int)((int64_t)kTiles * split / splits), t1 = (int)((int64_t)kTiles * (split + 1) / splits);
  const int *pt = table + r * kReqPages;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & 15;
  u32x4 acc = {0, 0, 0, 0};
  for (int t = t0 + wave; t < t1; t += 4) {
    u32x4 v[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int key = t * kTile + 4 * i + lane / 16;
      if (key < kKvLen) {
        const int page = pt[2 * t + i / 4];
        const int64_t off = (((int64_t)page * kPage + (4 * i) % 16 + lane / 16) * kHkv + h) * kD + c * 8;
        v[2 * i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(kp + off));
        v[2 * i + 1] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(vp + off));
      } else {
        v[2 * i] = u32x4{0, 0, 0, 0};
        v[2 * i + 1] = u32x4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) acc ^= v[e];
  }
  keep(acc, sink);
}

typedef __amdgpu_buffer_rsrc_t BufRsrc;
typedef __attribute__((address_space(3))) void lds_void_t;

// Wave w of a workgroup copies tiles t0 + w, t0 + w + 4, ... of its
// (request, KV head): instruction i moves key rows 4 i .. 4 i + 3 (16 lanes
// per 256-byte row) of K, then of V, into the wave's 16 KiB LDS area; the
// wave waits for the tile and folds 16 bytes of it.
__global__ __launch_bounds__(256) void dma_kernel(const uint16_t *kp, const uint16_t *vp, const int *table,
                                                  int splits, u32x4 *sink) {
  __shared__ __attribute__((aligned(1024))) char lds[4 * 16384];
  const int w = blockIdx.x;
  const int split = w % splits, pair = w / splits;
  const int h = pair % kHkv, r = pair / kHkv;
  const int t0 = (int)((int64_t)kTiles * split / splits), t1 = (int)((int64_t)kTiles * (split + 1) / splits);
  const int *pt = table + r * kReqPages;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  char *const mine = lds + wave * 16384;
  const int64_t row_el = (int64_t)kHkv * kD;
  u32x4 acc = {0, 0, 0, 0};
  for (int t = t0 + wave; t < t1; t += 4) {
    const int pa = pt[2 * t];
    const int pb = t * kTile + 16 < kKvLen ? pt[2 * t + 1] : pa;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k0 = t * kTile + 4 * i;                  // first key of the instruction
      const int half = (4 * i) / 16;
      const int page = half ? pb : pa;
      const int valid = k0 < kKvLen ? kKvLen - (k0 - (4 * i) % 16) : 0;   // tokens of this page in range
      const int nv = valid > kPage ? kPage : valid;
      const int bytes = nv > 0 ? (int)(((int64_t)(nv - 1) * row_el + kD) * 2) : 0;
      const int64_t pbase = ((int64_t)page * kPage * kHkv + h) * kD;
      const int voff = (int)((((4 * i) % 16 + lane / 16) * row_el + (lane % 16) * 8) * 2);
      const BufRsrc rk = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(kp + pbase), (short)0, bytes, 0x00020000);
      const BufRsrc rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(vp + pbase), (short)0, bytes, 0x00020000);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void_t *)(mine + i * 1024), 16, voff, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void_t *)(mine + 8192 + i * 1024), 16, voff, 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));   // vmcnt(0)
    acc ^= *reinterpret_cast<volatile u32x4 *>(mine + lane * 16);
  }
  keep(acc, sink);
}

template <typename L>
float time_ms(L &&launch, int reps) {
  hipEvent_t a, b;
  (void)hipEventCreate(&a);
  (void)hipEventCreate(&b);
  for (int i = 0; i < 3; ++i) launch();
  (void)hipEventRecord(a, 0);
  for (int i = 0; i < reps; ++i) launch();
  (void)hipEventRecord(b, 0);
  (void)hipEventSynchronize(b);
  float ms = 0.f;
  (void)hipEventElapsedTime(&ms, a, b);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  return ms / reps;
}

}  // namespace

int main() {
  // Page table: request r holds kSel distinct cartridges (a fixed LCG draw),
  // their pages in order, then its own pages after the cartridge region.
  std::vector<int> table((size_t)kReqs * kReqPages);
  uint64_t s = 0x2545F4914F6CDD1DULL;
  auto next = [&]() {
    s = s * 6364136223846793005ULL + 1442695040888963407ULL;
    return (int)((s >> 33) % kCarts);
  };
  for (int r = 0; r < kReqs; ++r) {
    int sel[kSel];
    for (int i = 0; i < kSel; ++i) {
      bool dup;
      do {
        sel[i] = next();
        dup = false;
        for (int j = 0; j < i; ++j) dup |= sel[j] == sel[i];
      } while (dup);
    }
    int *pt = &table[(size_t)r * kReqPages];
    for (int i = 0; i < kSel; ++i)
      for (int j = 0; j < kCartPages; ++j) pt[i * kCartPages + j] = sel[i] * kCartPages + j;
    for (int j = 0; j < kOwnPages; ++j) pt[kSel * kCartPages + j] = kCarts * kCartPages + r * kOwnPages + j;
  }
  for (int x : table)
    if (x < 0 || x >= kPages) {
      printf("page id out of range\n");
      return 1;
    }

  uint16_t *kp, *vp;
  int *dt;
  u32x4 *sink;
  const size_t pool_bytes = (size_t)kPoolElems * 2;
  CHECK(hipMalloc(&kp, 2 * pool_bytes));
  vp = kp + kPoolElems;
  CHECK(hipMemset(kp, 0x3c, 2 * pool_bytes));
  CHECK(hipMalloc(&dt, table.size() * sizeof(int)));
  CHECK(hipMemcpy(dt, table.data(), table.size() * sizeof(int), hipMemcpyHostToDevice));
  const int max_wg = kReqs * kHkv * 8;
  CHECK(hipMalloc(&sink, (size_t)std::max(max_wg, 4096) * 256 * sizeof(u32x4)));

  const double dec_bytes = (double)kReqs * kHkv * kKvLen * kD * 2 * 2;   // K and V, per request
  printf("pool %.3f GB (K and V), decode bytes %.4f GB, %d requests x %d KV heads x %d keys\n",
         2.0 * pool_bytes / 1e9, dec_bytes / 1e9, kReqs, kHkv, kKvLen);

  const int64_t n16 = (int64_t)(2 * pool_bytes / 16);
  for (int grid : {1024, 2048, 4096}) {
    const float ms = time_ms([&] { hipLaunchKernelGGL(seq_kernel<4>, dim3(grid), dim3(256), 0, 0,
                                                      (const u32x4 *)kp, n16, sink); }, 20);
    CHECK(hipGetLastError());
    printf("seq     grid %5d U 4: %.4f ms  %.0f GB/s\n", grid, ms, 2.0 * pool_bytes / ms / 1e6);
  }
  auto run_pages = [&](auto UC, int splits) {
    constexpr int U = decltype(UC)::value;
    const int grid = kReqs * kHkv * splits;
    const float ms = time_ms([&] { hipLaunchKernelGGL(pages_kernel<U>, dim3(grid), dim3(256), 0, 0, kp, vp,
                                                      dt, splits, sink); }, 20);
    printf("pages   grid %5d U %d: %.4f ms  %.0f GB/s of decode bytes\n", grid, U, ms, dec_bytes / ms / 1e6);
  };
  for (int splits : {1, 2, 4, 8}) {
    run_pages(std::integral_constant<int, 1>{}, splits);
    run_pages(std::integral_constant<int, 2>{}, splits);
    run_pages(std::integral_constant<int, 4>{}, splits);
  }
  for (int splits : {1, 2, 4}) {
    const int grid = kReqs * kHkv * splits;
    const float ms = time_ms([&] { hipLaunchKernelGGL(wave_kernel, dim3(grid), dim3(256), 0, 0, kp, vp, dt, splits,
                                                      sink); }, 20);
    printf("wave    grid %5d    : %.4f ms  %.0f GB/s of decode bytes\n", grid, ms, dec_bytes / ms / 1e6);
  }
  for (int splits : {1, 2, 4}) {
    const int grid = kReqs * kHkv * splits;
    const float ms = time_ms([&] { hipLaunchKernelGGL(dma_kernel, dim3(grid), dim3(256), 0, 0, kp, vp, dt, splits,
                                                      sink); }, 20);
    printf("dma     grid %5d    : %.4f ms  %.0f GB/s of decode bytes\n", grid, ms, dec_bytes / ms / 1e6);
  }
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  CHECK(hipFree(kp));
  CHECK(hipFree(dt));
  CHECK(hipFree(sink));
  return 0;
}
