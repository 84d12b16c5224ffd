// Measurement probe (not part of libcas): the cost of accumulating dQ with
// fp32 atomic adds from a key-stationary backward pass, on the 16 x 2,048
// workload (batch 2, 8 KV heads, 4 query heads per KV head, d = 128, 2,048
// queries and a 32,768-token prefix per row).
//
// A fused dK/dV/dQ pass would have every key workgroup add its dQ partial
// dS K (64 rows x 128 channels fp32, 32 KiB) into each 64-row query block of
// its (row, KV head): 16 groups x 128 query blocks, and 264 workgroups per
// group with 128-key tiles (32,768 + 2,048 keys / 128, self tiles rounded
// up) or 66 with 512-key super-tiles. The probe issues exactly that stream
// of adds, each workgroup starting at a different block so that the adds
// into one block are spread in time, and times it with HIP events; plain
// stores of the same pattern give the memory system's rate without atomics.
// Every mode checks its result on the host.
//
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       paper_2606_04557_amd/probes/atomic_dq_stream.hip -o atomic_dq_stream
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

namespace {

constexpr int kGroups = 16;            // (row, KV head) pairs
constexpr int kBlocks = 128;           // 64-row query blocks per group
constexpr int kBlockFloats = 64 * 128;  // one fp32 dQ block
constexpr int kThreads = 256;

enum Mode { kAtomicAgent = 0, kAtomicWorkgroup = 1, kStore = 2 };

// Workgroup w adds (or stores) 1.0 into every element of every block of its
// group, starting at block (its tile) mod kBlocks. With xcd_affine, the
// workgroups of one group run on one XCD (dispatch is round-robin over 8).
template <int MODE>
__global__ __launch_bounds__(kThreads) void stream(float *acc, int tiles, int xcd_affine) {
  const int w = blockIdx.x;
  int grp, tile;
  if (xcd_affine) {
    const int x = w % 8, i = w / 8;
    grp = x * 2 + (i % 2);
    tile = i / 2;
  } else {
    grp = w % kGroups;
    tile = w / kGroups;
  }
  if (tile >= tiles) return;
  float *base = acc + (size_t)grp * kBlocks * kBlockFloats;
  for (int k = 0; k < kBlocks; ++k) {
    float *b = base + (size_t)((k + tile) % kBlocks) * kBlockFloats;
#pragma unroll 4
    for (int e = threadIdx.x; e < kBlockFloats; e += kThreads) {
      if constexpr (MODE == kAtomicAgent)
        __hip_atomic_fetch_add(b + e, 1.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else if constexpr (MODE == kAtomicWorkgroup)
        __hip_atomic_fetch_add(b + e, 1.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      else
        b[e] = 1.0f;
    }
  }
}

#define CHECK(x)                                                                          \
  do {                                                                                    \
    hipError_t e_ = (x);                                                                  \
    if (e_ != hipSuccess) {                                                               \
      std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));                 \
      std::exit(1);                                                                       \
    }                                                                                     \
  } while (0)

void launch(int mode, int grid, float *acc, int tiles, int aff) {
  if (mode == kAtomicAgent) hipLaunchKernelGGL(stream<kAtomicAgent>, dim3(grid), dim3(kThreads), 0, 0, acc, tiles, aff);
  if (mode == kAtomicWorkgroup)
    hipLaunchKernelGGL(stream<kAtomicWorkgroup>, dim3(grid), dim3(kThreads), 0, 0, acc, tiles, aff);
  if (mode == kStore) hipLaunchKernelGGL(stream<kStore>, dim3(grid), dim3(kThreads), 0, 0, acc, tiles, aff);
}

}  // namespace

int main() {
  const size_t n = (size_t)kGroups * kBlocks * kBlockFloats;
  float *acc = nullptr;
  CHECK(hipMalloc(&acc, n * sizeof(float)));
  hipEvent_t t0, t1;
  CHECK(hipEventCreate(&t0));
  CHECK(hipEventCreate(&t1));
  std::vector<float> h(n);
  const char *names[] = {"atomic add, agent scope", "atomic add, workgroup scope", "plain store"};
  int bad = 0;
  for (int tiles : {264, 66}) {
    const int grid = kGroups * tiles;
    const double bytes = (double)grid * kBlocks * kBlockFloats * sizeof(float);
    for (int mode = 0; mode < 3; ++mode) {
      for (int aff = 0; aff < 2; ++aff) {
        if (mode == kStore && aff) continue;
        float best = 1e30f;
        for (int rep = 0; rep < 3; ++rep) {
          CHECK(hipMemset(acc, 0, n * sizeof(float)));
          CHECK(hipDeviceSynchronize());
          CHECK(hipEventRecord(t0));
          launch(mode, grid, acc, tiles, aff);
          CHECK(hipGetLastError());
          CHECK(hipEventRecord(t1));
          CHECK(hipEventSynchronize(t1));
          float ms = 0.0f;
          CHECK(hipEventElapsedTime(&ms, t0, t1));
          best = ms < best ? ms : best;
        }
        CHECK(hipMemcpy(h.data(), acc, n * sizeof(float), hipMemcpyDeviceToHost));
        const float want = mode == kStore ? 1.0f : (float)tiles;
        size_t wrong = 0;
        for (size_t i = 0; i < n; ++i) wrong += h[i] != want;
        bad += wrong != 0;
        std::printf("%3d keys per workgroup, %-28s xcd_affine %d: %8.3f ms for %6.2f GB, %7.1f GB/s%s\n",
                    tiles == 264 ? 128 : 512, names[mode], aff, best, bytes / 1e9, bytes / best / 1e6,
                    wrong ? "  WRONG RESULT" : "");
        std::fflush(stdout);
      }
    }
  }
  CHECK(hipFree(acc));
  return bad ? 1 : 0;
}
