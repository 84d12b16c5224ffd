// Forward of multi-cartridge prefix attention on gfx950.
//
// One workgroup owns 256 packed query rows (4 waves x 64) of one (batch row,
// kv head) and walks that row's key axis -- every cartridge segment in table
// order, then the causal self keys -- in 64-key tiles staged through LDS. The
// GQA group's query heads share each tile. Per tile and wave:
//   S^T = K Q^T   (MFMA; K from LDS in row layout, Q held in registers)
//   online softmax on S^T (a lane owns one query column: row max/sum are
//   lane-local plus one exchange with the partner lane 32 away)
//   O^T += V^T P^T (MFMA; V from LDS, P^T straight from the S^T registers)
// This is the fp32 path (v_mfma_f32_32x32x2f32, no down-conversion); bf16
// runs the kernels of cas_bf16.hip.
// Segment tiles stop at segment ends, so a ragged tail is the only masked
// prefix tile; self tiles are masked only where they cross the diagonal.
// With splits > 1 each workgroup takes a contiguous share of the key tiles
// and writes a normalised partial O and its LSE, merged afterwards.
#include <algorithm>

#include "cas_device.h"

namespace cas {

template <int D>
__global__ __launch_bounds__(kThreads) void fwd_kernel(FwdParams p) {
  using T = float;
  using M = Mma<T>;
  using Frag = typename M::Frag;
  constexpr int NSTEP = D / M::kStep;
  constexpr int QS = kRowsPerWave / 32;
  constexpr int KT = kKeyTile;
  constexpr int NSUB = KT / 32;
  constexpr int DT = D / 32;
  constexpr int RS = lds_row_stride<T, D>();

  __shared__ __attribute__((aligned(16))) T k_lds[KT * RS];
  __shared__ __attribute__((aligned(16))) T v_lds[KT * RS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = lane >> 5, n = lane & 31;
  int bid = blockIdx.x;
  const int qblk = bid % p.nqblk;
  bid /= p.nqblk;
  const int kvh = bid % p.Hkv;
  bid /= p.Hkv;
  const int split = bid % p.splits;
  const int b = bid / p.splits;

  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g;
  const DevRow row = p.rows[b];
  const int tok0 = row.tok0, len = row.len, nrows = len * g;
  const int wg_row0 = qblk * kRowsPerWg;
  if (wg_row0 >= nrows) return;   // grid sized for the longest row
  const int wg_row1 = min(nrows, wg_row0 + kRowsPerWg);
  const int row0 = wg_row0 + wave * kRowsPerWave;
  const bool wave_active = row0 < nrows;
  const int wave_t_lo = row0 / g;
  const int wave_t_hi = (min(row0 + kRowsPerWave, nrows) - 1) / g;
  const int wg_t_hi = (wg_row1 - 1) / g;
  const float c = p.scale_log2;

  Frag qf[QS][NSTEP];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int r = row0 + 32 * qs + n;
    if (r < nrows) {
      const int t = r / g, hh = r - t * g;
      const T *rp = (const T *)p.q + (((int64_t)tok0 + t) * Hq + kvh * g + hh) * D;
#pragma unroll
      for (int st = 0; st < NSTEP; ++st) qf[qs][st] = global_frag<T>(rp, st, G);
    } else {
#pragma unroll
      for (int st = 0; st < NSTEP; ++st) qf[qs][st] = M::zero();
    }
  }

  f32x16 oacc[DT][QS];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) oacc[dt][qs] = zero16();
  float m_run[QS], l_run[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    m_run[qs] = -INFINITY;
    l_run[qs] = 0.0f;
  }

  const int ptiles = row.prefix_tiles;
  const int ntiles = ptiles + wg_t_hi / KT + 1;
  const int tb = (int)((int64_t)ntiles * split / p.splits);
  const int te = (int)((int64_t)ntiles * (split + 1) / p.splits);
  int seg = row.seg_begin;

  for (int tile = tb; tile < te; ++tile) {
    const T *kp;
    const T *vp;
    int64_t st;
    int nvalid;
    int self0 = -1;
    if (tile < ptiles) {
      for (;;) {
        const DevSeg sd = p.segs[seg];
        if (tile < sd.tile_begin + (sd.len + KT - 1) / KT) break;
        ++seg;
      }
      const DevSeg sd = p.segs[seg];
      const int key0 = (tile - sd.tile_begin) * KT;
      kp = (const T *)sd.k + kvh * sd.stride_head + (int64_t)key0 * sd.stride_tok;
      vp = (const T *)sd.v + kvh * sd.stride_head + (int64_t)key0 * sd.stride_tok;
      st = sd.stride_tok;
      nvalid = min(KT, sd.len - key0);
    } else {
      self0 = (tile - ptiles) * KT;
      kp = (const T *)p.k_self + (((int64_t)tok0 + self0) * Hkv + kvh) * D;
      vp = (const T *)p.v_self + (((int64_t)tok0 + self0) * Hkv + kvh) * D;
      st = (int64_t)Hkv * D;
      nvalid = min(KT, len - self0);
    }
    __syncthreads();
    load_rows<T, D, KT>(k_lds, [&](int r) { return kp + r * st; }, nvalid, tid);
    load_rows<T, D, KT>(v_lds, [&](int r) { return vp + r * st; }, nvalid, tid);
    __syncthreads();

    if (!wave_active) continue;
    if (self0 >= 0 && self0 > wave_t_hi) continue;
    const bool need_mask = (nvalid < KT) || (self0 >= 0 && self0 + KT - 1 > wave_t_lo);

    f32x16 sacc[NSUB][QS];
#pragma unroll
    for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) sacc[sub][qs] = zero16();
#pragma unroll
    for (int stp = 0; stp < NSTEP; ++stp) {
      Frag kf[NSUB];
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub) kf[sub] = row_frag<T, D>(k_lds, 32 * sub + n, stp, G);
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) sacc[sub][qs] = M::run(kf[sub], qf[qs][stp], sacc[sub][qs]);
    }

#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      const int t = (row0 + 32 * qs + n) / g;
      float mx = -INFINITY;
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          float x = sacc[sub][qs][j];
          if (need_mask) {
            const int key = 32 * sub + crow(j, G);
            const bool ok = key < nvalid && (self0 < 0 || self0 + key <= t);
            x = ok ? x : -INFINITY;
            sacc[sub][qs][j] = x;
          }
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, xor32(mx));
      const float m_new = fmaxf(m_run[qs], mx * c);
      const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
      const float alpha = exp2f(m_run[qs] - m_use);
      float ls = 0.0f;
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float pv = exp2f(fmaf(sacc[sub][qs][j], c, -m_use));
          sacc[sub][qs][j] = pv;
          ls += pv;
        }
      l_run[qs] = l_run[qs] * alpha + ls;
      m_run[qs] = m_new;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt][qs] *= alpha;
    }

#pragma unroll
    for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
      for (int s = 0; s < 16; ++s)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const float a = trans_frag_f32<D>(v_lds, sub, s, G, dt * 32 + n);
#pragma unroll
          for (int qs = 0; qs < QS; ++qs) oacc[dt][qs] = M::run(a, sacc[sub][qs][s], oacc[dt][qs]);
        }
  }

#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const float lt = l_run[qs] + xor32(l_run[qs]);
    const int r = row0 + 32 * qs + n;
    if (r >= nrows) continue;
    const int t = r / g, hh = r - t * g, h = kvh * g + hh;
    if (p.splits == 1) {
      const float inv = 1.0f / lt;
      T *op = (T *)p.o + (((int64_t)tok0 + t) * Hq + h) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          store4(op + dt * 32 + jj * 8 + G * 4, oacc[dt][qs][jj * 4 + 0] * inv,
                 oacc[dt][qs][jj * 4 + 1] * inv, oacc[dt][qs][jj * 4 + 2] * inv,
                 oacc[dt][qs][jj * 4 + 3] * inv);
      if (G == 0 && p.lse != nullptr)
        p.lse[(int64_t)row.lse0 + (int64_t)h * p.lse_hs + t] = (m_run[qs] + log2f(lt)) * kLn2;
    } else {
      const int64_t prow = split * p.plane + (int64_t)tok0 * Hq + kvh * nrows + r;
      const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
      float *op = p.part_o + prow * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          store4(op + dt * 32 + jj * 8 + G * 4, oacc[dt][qs][jj * 4 + 0] * inv,
                 oacc[dt][qs][jj * 4 + 1] * inv, oacc[dt][qs][jj * 4 + 2] * inv,
                 oacc[dt][qs][jj * 4 + 3] * inv);
      if (G == 0) p.part_lse[prow] = lt > 0.0f ? (m_run[qs] + log2f(lt)) * kLn2 : -INFINITY;
    }
  }
}

// LSE-weighted combination of split partials:
//   LSE = log sum_s exp(LSE_s),  O = sum_s exp(LSE_s - LSE) O_s.
// One thread per 4 channels of a packed row; grid.y is the batch row.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void fwd_merge_kernel(MergeParams p) {
  constexpr int CPR = D / 4;
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int b = blockIdx.y;
  const DevRow row = p.rows[b];
  const int nrows = row.len * p.g;
  const int64_t rb = idx / CPR;          // kvh * nrows + r
  const int c4 = (int)(idx % CPR);
  if (rb >= (int64_t)p.Hkv * nrows) return;
  const int64_t plane = p.plane;
  const int64_t R = (int64_t)row.tok0 * p.Hkv * p.g + rb;
  float mx = -INFINITY;
  for (int s = 0; s < p.splits; ++s) mx = fmaxf(mx, p.part_lse[s * plane + R]);
  float w_sum = 0.0f;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int s = 0; s < p.splits; ++s) {
    const float ls = p.part_lse[s * plane + R];
    const float w = (ls == -INFINITY) ? 0.0f : expf(ls - mx);
    w_sum += w;
    const f32x4 v = *reinterpret_cast<const f32x4 *>(p.part_o + (s * plane + R) * D + c4 * 4);
    acc += w * v;
  }
  const float inv = 1.0f / w_sum;
  const int kvh = (int)(rb / nrows), r = (int)(rb % nrows);
  const int t = r / p.g, h = kvh * p.g + (r - t * p.g);
  const int Hq = p.Hkv * p.g;
  T *op = (T *)p.o + (((int64_t)row.tok0 + t) * Hq + h) * D + c4 * 4;
  store4(op, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  if (c4 == 0 && p.lse != nullptr) p.lse[(int64_t)row.lse0 + (int64_t)h * p.lse_hs + t] = mx + logf(w_sum);
}

template <int D>
static hipError_t launch_fwd_t(const FwdParams &p, hipStream_t s) {
  const int64_t grid = (int64_t)p.nqblk * p.Hkv * p.splits * p.B;
  hipLaunchKernelGGL((fwd_kernel<D>), dim3((unsigned)grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_fwd(const FwdParams &p, DType dt, int D, hipStream_t s) {
  if (dt == kBF16) return launch_fwd_bf16(p, D, s);
  return D == 64 ? launch_fwd_t<64>(p, s) : launch_fwd_t<128>(p, s);
}

template <typename T, int D>
static hipError_t launch_merge_t(const MergeParams &p, hipStream_t s) {
  const int64_t n = (int64_t)p.Hkv * p.nrows_max * (D / 4);
  const dim3 grid((unsigned)((n + kThreads - 1) / kThreads), (unsigned)p.B);
  hipLaunchKernelGGL((fwd_merge_kernel<T, D>), grid, dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

// Launch-table upload: copies `bytes` from pinned host memory to the device
// workspace (both 16-byte aligned), 16 bytes per thread and the last
// bytes % 16 one by one. A kernel on the launch stream instead of a
// copy-engine transfer, so the kernels that read the tables follow it
// without a hand-over between engines.
__global__ __launch_bounds__(256) void table_upload_kernel(char *dst, const char *src, int64_t bytes) {
  const int64_t n16 = bytes / 16;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (int64_t)gridDim.x * 256)
    reinterpret_cast<uint4 *>(dst)[i] = reinterpret_cast<const uint4 *>(src)[i];
  if (blockIdx.x == 0 && threadIdx.x < (unsigned)(bytes - n16 * 16)) dst[n16 * 16 + threadIdx.x] = src[n16 * 16 + threadIdx.x];
}

hipError_t launch_table_upload(void *dst, const void *src, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>(((int64_t)bytes / 16 + 255) / 256, 64));
  hipLaunchKernelGGL(table_upload_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (char *)dst, (const char *)src,
                     (int64_t)bytes);
  return hipGetLastError();
}

hipError_t launch_fwd_merge(const MergeParams &p, DType dt, int D, hipStream_t s) {
  if (dt == kBF16) return D == 64 ? launch_merge_t<__bf16, 64>(p, s) : launch_merge_t<__bf16, 128>(p, s);
  return D == 64 ? launch_merge_t<float, 64>(p, s) : launch_merge_t<float, 128>(p, s);
}

}  // namespace cas
