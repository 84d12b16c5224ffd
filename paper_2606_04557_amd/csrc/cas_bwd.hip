// Backward of multi-cartridge prefix attention on gfx950: the statistics
// pass for both dtypes, the fp32 dK/dV and dQ passes (v_mfma_f32_32x32x2f32,
// no down-conversion; bf16 runs the kernels of cas_bf16.hip) and the dQ
// split reduction for both dtypes.
//
// Three passes, all recomputing P from the stored row LSE:
//   bwd_pre:  D = rowsum(dO * O) and LSE*log2(e) per packed row (fp32).
//   dkdv:     key-stationary. A workgroup owns 128 keys (4 waves x 32) of one
//             distinct cartridge (or of one row's self keys) and one kv head;
//             it loops over every query row of the GQA group in every batch
//             row that references the cartridge, with Q/dO blocks staged
//             through LDS:
//               S = Q K^T, dP = dO V^T        (K, V held in registers)
//               P = exp2(S c - LSE2), dS = P (dP - D)
//               dV^T += dO^T P, dK^T += Q^T dS  (P, dS straight from the C
//                                                registers; Q/dO from LDS)
//             The sums stay in registers, so each key's gradient is written
//             once, to the owning segment's buffer, with no atomics; a
//             cartridge referenced by several rows accumulates all of them.
//   dq:       query-stationary, like the forward: per key tile
//               S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - D),
//               dQ^T += K^T dS^T
//             with optional key-axis splits whose fp32 partials are summed.
#include "cas_device.h"

namespace cas {

// 16 lanes per packed row; grid.y is the batch row.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void bwd_pre_kernel(PreParams p) {
  constexpr int LPR = 16;            // lanes per packed row
  constexpr int CPL = D / LPR;       // channels per lane
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int b = blockIdx.y;
  const DevRow row = p.rows[b];
  const int nrows = row.len * p.g;
  const int64_t rb = gid / LPR;      // kvh * nrows + r
  const int li = (int)(gid % LPR);
  const bool live = rb < (int64_t)p.Hkv * nrows;
  const int Hq = p.Hkv * p.g;
  float acc = 0.0f;
  int h = 0, t = 0;
  if (live) {
    const int kvh = (int)(rb / nrows), r = (int)(rb % nrows);
    t = r / p.g;
    h = kvh * p.g + (r - t * p.g);
    const int64_t off = (((int64_t)row.tok0 + t) * Hq + h) * D + li * CPL;
    const T *op = (const T *)p.o + off;
    const T *dp = (const T *)p.d_o + off;
#pragma unroll
    for (int i = 0; i < CPL; ++i) acc += to_f32(op[i]) * to_f32(dp[i]);
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, LPR);
  if (live && li == 0) {
    const int64_t R = (int64_t)row.tok0 * Hq + rb;
    p.nd[R] = -acc;
    p.lse2[R] = p.lse[(int64_t)row.lse0 + (int64_t)h * p.lse_hs + t] * kLog2e;
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void dkdv_kernel(DkdvParams p) {
  using T = float;
  using M = Mma<T>;
  using Frag = typename M::Frag;
  constexpr int NSTEP = D / M::kStep;
  constexpr int QB = kDkdvQBlock;
  constexpr int QSUB = QB / 32;
  constexpr int DT = D / 32;
  constexpr int RS = lds_row_stride<T, D>();

  __shared__ __attribute__((aligned(16))) T q_row[QB * RS];
  __shared__ __attribute__((aligned(16))) T do_row[QB * RS];
  __shared__ float lse2_l[QB];
  __shared__ float nd_l[QB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = lane >> 5, n = lane & 31;
  const DevWg wg = p.order[blockIdx.x];
  const int tile = wg.tile, kvh = wg.kvh;
  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g;
  const float c = p.scale_log2;

  const T *kbase;
  const T *vbase;
  T *dkp;
  T *dvp;
  int64_t st;
  int klen, key0, use_b = 0, use_e = 1;
  const bool self = tile >= p.cart_tiles;
  int self_b = 0;
  if (!self) {
    int lo = 0, hi = p.n_carts - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (p.carts[mid].tile_begin <= tile) lo = mid; else hi = mid - 1;
    }
    const DevCart cd = p.carts[lo];
    key0 = (tile - cd.tile_begin) * kDkdvKeyTile;
    klen = cd.len;
    kbase = (const T *)cd.k + kvh * cd.stride_head;
    vbase = (const T *)cd.v + kvh * cd.stride_head;
    dkp = cd.dk ? (T *)cd.dk + kvh * cd.stride_head : nullptr;
    dvp = cd.dv ? (T *)cd.dv + kvh * cd.stride_head : nullptr;
    st = cd.stride_tok;
    use_b = cd.use_begin;
    use_e = cd.use_end;
  } else {
    const int rel = tile - p.cart_tiles;
    self_b = rel / p.self_tiles;
    key0 = (rel % p.self_tiles) * kDkdvKeyTile;
    const DevRow sr = p.rows[self_b];
    klen = sr.len;
    if (key0 >= klen) return;   // grid sized for the longest row
    const int64_t base = ((int64_t)sr.tok0 * Hkv + kvh) * D;
    kbase = (const T *)p.k_self + base;
    vbase = (const T *)p.v_self + base;
    dkp = p.dk_self ? (T *)p.dk_self + base : nullptr;
    dvp = p.dv_self ? (T *)p.dv_self + base : nullptr;
    st = (int64_t)Hkv * D;
  }
  const int wkey0 = key0 + wave * kDkdvKeysPerWave;
  const int my_key = wkey0 + n;
  const bool key_ok = my_key < klen;
  const bool wave_has_keys = wkey0 < klen;

  Frag kf[NSTEP], vf[NSTEP];
#pragma unroll
  for (int s = 0; s < NSTEP; ++s) {
    kf[s] = key_ok ? global_frag<T>(kbase + my_key * st, s, G) : M::zero();
    vf[s] = key_ok ? global_frag<T>(vbase + my_key * st, s, G) : M::zero();
  }
  f32x16 dk[DT], dv[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    dk[dt] = zero16();
    dv[dt] = zero16();
  }

  const int qb0 = self ? (key0 * g) / QB : 0;
  for (int u = use_b; u < use_e; ++u) {
    const int b = self ? self_b : p.uses[u];
    const DevRow rw = p.rows[b];
    const int nrows = rw.len * g;
    const int nqb = (nrows + QB - 1) / QB;
    const T *qb_base = (const T *)p.q + ((int64_t)rw.tok0 * Hq + kvh * g) * D;
    const T *dob_base = (const T *)p.d_o + ((int64_t)rw.tok0 * Hq + kvh * g) * D;
    const float *lse2_b = p.lse2 + (int64_t)rw.tok0 * Hq + (int64_t)kvh * nrows;
    const float *nd_b = p.nd + (int64_t)rw.tok0 * Hq + (int64_t)kvh * nrows;
    for (int qb = qb0; qb < nqb; ++qb) {
      const int r0 = qb * QB;
      const int nv = min(QB, nrows - r0);
      auto qptr = [&](int r) {
        const int rr = r0 + r, t = rr / g;
        return qb_base + ((int64_t)t * Hq + (rr - t * g)) * D;
      };
      auto doptr = [&](int r) {
        const int rr = r0 + r, t = rr / g;
        return dob_base + ((int64_t)t * Hq + (rr - t * g)) * D;
      };
      __syncthreads();
      load_rows<T, D, QB>(q_row, qptr, nv, tid);
      load_rows<T, D, QB>(do_row, doptr, nv, tid);
      if (tid < QB) {
        const int rr = r0 + tid;
        lse2_l[tid] = rr < nrows ? lse2_b[rr] : INFINITY;
        nd_l[tid] = rr < nrows ? nd_b[rr] : 0.0f;
      }
      __syncthreads();
      if (!wave_has_keys) continue;
      const int blk_t_lo = r0 / g, blk_t_hi = (r0 + nv - 1) / g;
      if (self && wkey0 > blk_t_hi) continue;
      const bool need_mask = self && (wkey0 + kDkdvKeysPerWave - 1 > blk_t_lo);

#pragma unroll
      for (int qs = 0; qs < QSUB; ++qs) {
        f32x16 sa = zero16(), dpa = zero16();
#pragma unroll
        for (int s = 0; s < NSTEP; ++s) {
          sa = M::run(row_frag<T, D>(q_row, 32 * qs + n, s, G), kf[s], sa);
          dpa = M::run(row_frag<T, D>(do_row, 32 * qs + n, s, G), vf[s], dpa);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int ql = 32 * qs + crow(j, G);
          float pv = exp2f(fmaf(sa[j], c, -lse2_l[ql]));
          if (need_mask) pv = (my_key <= (r0 + ql) / g) ? pv : 0.0f;
          pv = key_ok ? pv : 0.0f;
          const float ds = pv * (dpa[j] + nd_l[ql]);
          sa[j] = pv;
          dpa[j] = ds;
        }
#pragma unroll
        for (int s = 0; s < 16; ++s)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            dv[dt] = M::run(trans_frag_f32<D>(do_row, qs, s, G, dt * 32 + n), sa[s], dv[dt]);
            dk[dt] = M::run(trans_frag_f32<D>(q_row, qs, s, G, dt * 32 + n), dpa[s], dk[dt]);
          }
      }
    }
  }

  if (!key_ok) return;
  const float sc = p.scale;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d0 = dt * 32 + jj * 8 + G * 4;
      if (dkp)
        store4(dkp + my_key * st + d0, dk[dt][jj * 4 + 0] * sc, dk[dt][jj * 4 + 1] * sc,
               dk[dt][jj * 4 + 2] * sc, dk[dt][jj * 4 + 3] * sc);
      if (dvp)
        store4(dvp + my_key * st + d0, dv[dt][jj * 4 + 0], dv[dt][jj * 4 + 1], dv[dt][jj * 4 + 2],
               dv[dt][jj * 4 + 3]);
    }
}

template <int D>
__global__ __launch_bounds__(kThreads) void dq_kernel(DqParams p) {
  using T = float;
  using M = Mma<T>;
  using Frag = typename M::Frag;
  constexpr int NSTEP = D / M::kStep;
  constexpr int QS = kDqRowsPerWave / 32;
  constexpr int KT = kKeyTile;
  constexpr int NSUB = KT / 32;
  constexpr int DT = D / 32;
  constexpr int RS = lds_row_stride<T, D>();

  __shared__ __attribute__((aligned(16))) T k_row[KT * RS];
  __shared__ __attribute__((aligned(16))) T v_row[KT * RS];

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
  const int wg_row0 = qblk * kDqRowsPerWg;
  if (wg_row0 >= nrows) return;   // grid sized for the longest row
  const int wg_row1 = min(nrows, wg_row0 + kDqRowsPerWg);
  const int row0 = wg_row0 + wave * kDqRowsPerWave;
  const bool wave_active = row0 < nrows;
  const int wave_t_lo = row0 / g;
  const int wave_t_hi = (min(row0 + kDqRowsPerWave, nrows) - 1) / g;
  const int wg_t_hi = (wg_row1 - 1) / g;
  const float c = p.scale_log2;

  Frag qf[QS][NSTEP], df[QS][NSTEP];
  float lse2r[QS], ndr[QS];
  const int64_t pk = (int64_t)tok0 * Hq + (int64_t)kvh * nrows;
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int r = row0 + 32 * qs + n;
    if (r < nrows) {
      const int t = r / g, hh = r - t * g;
      const int64_t off = (((int64_t)tok0 + t) * Hq + kvh * g + hh) * D;
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) {
        qf[qs][s] = global_frag<T>((const T *)p.q + off, s, G);
        df[qs][s] = global_frag<T>((const T *)p.d_o + off, s, G);
      }
      lse2r[qs] = p.lse2[pk + r];
      ndr[qs] = p.nd[pk + r];
    } else {
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) {
        qf[qs][s] = M::zero();
        df[qs][s] = M::zero();
      }
      lse2r[qs] = INFINITY;
      ndr[qs] = 0.0f;
    }
  }
  f32x16 acc[DT][QS];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = zero16();

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
    load_rows<T, D, KT>(k_row, [&](int r) { return kp + r * st; }, nvalid, tid);
    load_rows<T, D, KT>(v_row, [&](int r) { return vp + r * st; }, nvalid, tid);
    __syncthreads();

    if (!wave_active) continue;
    if (self0 >= 0 && self0 > wave_t_hi) continue;
    const bool need_mask = (nvalid < KT) || (self0 >= 0 && self0 + KT - 1 > wave_t_lo);

#pragma unroll
    for (int sub = 0; sub < NSUB; ++sub) {
      f32x16 sa[QS], dpa[QS];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
        sa[qs] = zero16();
        dpa[qs] = zero16();
      }
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) {
        const Frag kfr = row_frag<T, D>(k_row, 32 * sub + n, s, G);
        const Frag vfr = row_frag<T, D>(v_row, 32 * sub + n, s, G);
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) {
          sa[qs] = M::run(kfr, qf[qs][s], sa[qs]);
          dpa[qs] = M::run(vfr, df[qs][s], dpa[qs]);
        }
      }
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
        const int t = (row0 + 32 * qs + n) / g;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          float pv = exp2f(fmaf(sa[qs][j], c, -lse2r[qs]));
          if (need_mask) {
            const int key = 32 * sub + crow(j, G);
            const bool ok = key < nvalid && (self0 < 0 || self0 + key <= t);
            pv = ok ? pv : 0.0f;
          }
          sa[qs][j] = pv * (dpa[qs][j] + ndr[qs]);
        }
      }
#pragma unroll
      for (int s = 0; s < 16; ++s)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const float a = trans_frag_f32<D>(k_row, sub, s, G, dt * 32 + n);
#pragma unroll
          for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = M::run(a, sa[qs][s], acc[dt][qs]);
        }
    }
  }

#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int r = row0 + 32 * qs + n;
    if (r >= nrows) continue;
    const int t = r / g, h = kvh * g + (r - t * g);
    if (p.splits == 1) {
      const float sc = p.scale;
      T *op = (T *)p.dq + (((int64_t)tok0 + t) * Hq + h) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          store4(op + dt * 32 + jj * 8 + G * 4, acc[dt][qs][jj * 4 + 0] * sc,
                 acc[dt][qs][jj * 4 + 1] * sc, acc[dt][qs][jj * 4 + 2] * sc,
                 acc[dt][qs][jj * 4 + 3] * sc);
    } else {
      const int64_t prow = split * p.plane + pk + r;
      float *op = p.part_dq + prow * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          store4(op + dt * 32 + jj * 8 + G * 4, acc[dt][qs][jj * 4 + 0], acc[dt][qs][jj * 4 + 1],
                 acc[dt][qs][jj * 4 + 2], acc[dt][qs][jj * 4 + 3]);
    }
  }
}

// One thread per 4 channels of a packed row; grid.y is the batch row.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void dq_reduce_kernel(DqReduceParams p) {
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
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int s = 0; s < p.splits; ++s)
    acc += *reinterpret_cast<const f32x4 *>(p.part_dq + (s * plane + R) * D + c4 * 4);
  const int kvh = (int)(rb / nrows), r = (int)(rb % nrows);
  const int t = r / p.g, h = kvh * p.g + (r - t * p.g);
  const int Hq = p.Hkv * p.g;
  T *op = (T *)p.dq + (((int64_t)row.tok0 + t) * Hq + h) * D + c4 * 4;
  store4(op, acc[0] * p.scale, acc[1] * p.scale, acc[2] * p.scale, acc[3] * p.scale);
}

template <typename T, int D>
static hipError_t launch_pre_t(const PreParams &p, hipStream_t s) {
  const int64_t n = (int64_t)p.Hkv * p.nrows_max * 16;
  hipLaunchKernelGGL((bwd_pre_kernel<T, D>), dim3((unsigned)((n + kThreads - 1) / kThreads), (unsigned)p.B),
                     dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_bwd_pre(const PreParams &p, DType dt, int D, hipStream_t s) {
  if (dt == kBF16) return D == 64 ? launch_pre_t<__bf16, 64>(p, s) : launch_pre_t<__bf16, 128>(p, s);
  return D == 64 ? launch_pre_t<float, 64>(p, s) : launch_pre_t<float, 128>(p, s);
}

template <int D>
static hipError_t launch_dkdv_t(const DkdvParams &p, int n_wg, hipStream_t s) {
  hipLaunchKernelGGL((dkdv_kernel<D>), dim3((unsigned)n_wg), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_dkdv(const DkdvParams &p, DType dt, int D, int n_wg, hipStream_t s) {
  if (dt == kBF16) return launch_dkdv_bf16(p, D, n_wg, s);
  return D == 64 ? launch_dkdv_t<64>(p, n_wg, s) : launch_dkdv_t<128>(p, n_wg, s);
}

template <int D>
static hipError_t launch_dq_t(const DqParams &p, hipStream_t s) {
  const int64_t grid = (int64_t)p.nqblk * p.Hkv * p.splits * p.B;
  hipLaunchKernelGGL((dq_kernel<D>), dim3((unsigned)grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_dq(const DqParams &p, DType dt, int D, hipStream_t s) {
  if (dt == kBF16) return launch_dq_bf16(p, D, s);
  return D == 64 ? launch_dq_t<64>(p, s) : launch_dq_t<128>(p, s);
}

template <typename T, int D>
static hipError_t launch_dq_reduce_t(const DqReduceParams &p, hipStream_t s) {
  const int64_t n = (int64_t)p.Hkv * p.nrows_max * (D / 4);
  hipLaunchKernelGGL((dq_reduce_kernel<T, D>), dim3((unsigned)((n + kThreads - 1) / kThreads), (unsigned)p.B),
                     dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_dq_reduce(const DqReduceParams &p, DType dt, int D, hipStream_t s) {
  if (dt == kBF16) return D == 64 ? launch_dq_reduce_t<__bf16, 64>(p, s) : launch_dq_reduce_t<__bf16, 128>(p, s);
  return D == 64 ? launch_dq_reduce_t<float, 64>(p, s) : launch_dq_reduce_t<float, 128>(p, s);
}

}  // namespace cas
