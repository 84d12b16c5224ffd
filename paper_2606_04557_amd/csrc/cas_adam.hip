// Optimizer step of the trainable cartridges: Adam with fp32 moments on bf16
// parameters (paper: Section "Optimization Dynamics", paragraphs "Optimizer"
// and "Per-cartridge LR warmup"; Kingma and Ba, Algorithm 1).
//
// One launch covers every cartridge's K and V: the host lists each tensor
// (with its learning rate after the per-cartridge warmup and its bias
// corrections) and cuts the unfrozen tokens into chunks of kAdamChunk
// tokens, one workgroup each. The step is elementwise and moves 22 bytes per
// element (bf16 parameter and gradient read, fp32 moments read and written,
// bf16 parameter written), so it is HBM-bound: every lane moves 16-byte
// pieces (8 parameters, 8 gradients, 2 x 8 moments) with no reuse.
//
// The file is compiled without floating-point contraction, so each
// operation rounds once in the order the API documents.
#include "cas_device.h"

namespace cas {

template <int D>
__global__ __launch_bounds__(256) void adam_bf16_kernel(AdamParams p) {
  constexpr int CPR = D / 8;   // 8-element pieces per (token, head) row
  const DevAdamChunk ck = load_const(p.chunks, (int)blockIdx.x);
  const DevAdamT t = load_const(p.tensors, ck.t);
  const int Hkv = p.Hkv;
  const int ntok = min(kAdamChunk, t.len - ck.tok0);
  const int pieces = ntok * Hkv * CPR;
  const float b1 = p.beta1, b2 = p.beta2, omb1 = p.omb1, omb2 = p.omb2, eps = p.eps;
  for (int i = threadIdx.x; i < pieces; i += 256) {
    const int r = i / CPR, c8 = i - r * CPR;
    const int tok = ck.tok0 + r / Hkv, h = r - (r / Hkv) * Hkv;
    const int64_t xo = (int64_t)tok * t.stride_tok + (int64_t)h * t.stride_head + c8 * 8;
    const int64_t mo = ((int64_t)tok * Hkv + h) * D + c8 * 8;
    bf16x8 x = *reinterpret_cast<const bf16x8 *>(t.x + xo);
    const bf16x8 g = *reinterpret_cast<const bf16x8 *>(t.g + xo);
    f32x4 m1[2], m2[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      m1[k] = *reinterpret_cast<const f32x4 *>(t.m1 + mo + 4 * k);
      m2[k] = *reinterpret_cast<const f32x4 *>(t.m2 + mo + 4 * k);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float gf = (float)g[e];
      float a = m1[e >> 2][e & 3], s = m2[e >> 2][e & 3];
      a = b1 * a + omb1 * gf;
      s = b2 * s + omb2 * (gf * gf);
      m1[e >> 2][e & 3] = a;
      m2[e >> 2][e & 3] = s;
      const float mhat = a / t.bc1;
      const float vhat = s / t.bc2;
      const float step = (t.lr * mhat) / (__builtin_sqrtf(vhat) + eps);
      x[e] = (__bf16)((float)x[e] - step);
    }
    *reinterpret_cast<bf16x8 *>(t.x + xo) = x;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      *reinterpret_cast<f32x4 *>(t.m1 + mo + 4 * k) = m1[k];
      *reinterpret_cast<f32x4 *>(t.m2 + mo + 4 * k) = m2[k];
    }
  }
}

hipError_t launch_adam_bf16(const AdamParams &p, int D, int n_chunks, hipStream_t s) {
  if (D == 64)
    hipLaunchKernelGGL(adam_bf16_kernel<64>, dim3((unsigned)n_chunks), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(adam_bf16_kernel<128>, dim3((unsigned)n_chunks), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace cas
