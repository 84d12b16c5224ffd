// Short-query / decode attention over a paged KV pool (forward only): the
// retrieved cartridges' pages, then the request's own pages, with the last
// n queries of the key sequence as the new tokens (paper: Section
// "Inference", paragraph "Cartridge RAG", and the appendix on cartridge
// sizes for the 16-token pages of the serving engine's KV cache).
//
// A decode step has very few query rows per (request, KV head) (n * g, e.g.
// 4) against thousands of keys, so the work is streaming K and V out of HBM.
// One workgroup takes a block of up to 32 packed rows of one (request, KV
// head) and a range of 32-key tiles (the host splits a request's key axis
// so the whole GPU streams; partials are merged by their LSE). Its four waves
// work independently on every fourth tile of the range, each with its own
// double-buffered LDS tiles filled by direct buffer->LDS copies whose
// addresses come from the page table (one scalar load per page), so no wave
// ever waits on another until the end, where the four partial softmax states
// are combined through LDS. Per tile and wave: S^T = K Q^T (MFMA, K rows
// from LDS, Q in registers), an online-softmax update, and O^T += V^T P^T
// (MFMA, V^T by transposed LDS reads, P straight from the score registers).
#include "cas_device.h"

namespace cas {

namespace {

constexpr int kDecWaves = 4;

template <int D>
__global__ __launch_bounds__(kDecWaves * 64) void decode_bf16_kernel(DecodeParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int TB = kDecTile * D * 2;        // bytes of one 32-key tile
  constexpr int CPR = D / 8;                  // 16-byte chunks per key row
  constexpr int RPI = 64 / CPR;               // key rows per copy instruction
  constexpr int NI = kDecTile / RPI;          // copy instructions per tile (K or V)
  static_assert(kDecTile % RPI == 0 && 16 % RPI == 0, "copy instructions stay within a page");
  // Per wave: two stages of (K tile, V tile).
  __shared__ __attribute__((aligned(1024))) char smem[kDecWaves * 4 * TB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = lane >> 5, n = lane & 31;
  const DevDecodeWork w = load_const(p.work, (int)blockIdx.x);
  const DevDecodeReq rq = load_const(p.reqs, w.b);
  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g, P = p.page_size;
  const int kvh = __builtin_amdgcn_readfirstlane(w.kvh);
  const int kv_len = __builtin_amdgcn_readfirstlane(rq.kv_len);
  const int nrows = rq.n * g;
  const int my_row = w.row0 + n;
  const bool row_ok = my_row < nrows;
  const int my_i = my_row / g;                            // query index within the request
  const int my_h = kvh * g + (my_row - my_i * g);
  // Last key this row sees (rows past the block's end see every key: their
  // Q is zero and nothing of theirs is stored).
  const int my_lim = row_ok ? kv_len - rq.n + my_i : kv_len - 1;
  const float c = p.scale_log2;
  char *const wbase = smem + wave * 4 * TB;

  bf16x8 qf[NSTEP];
  if (row_ok) {
    const __bf16 *qp = (const __bf16 *)p.q + ((int64_t)(rq.q0 + my_i) * Hq + my_h) * D;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) qf[st] = *reinterpret_cast<const bf16x8 *>(qp + st * 16 + G * 8);
  } else {
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) qf[st] = Mma<__bf16>::zero();
  }
  // Tile copies are waited for with partial vmcnt counts, which must not
  // include these loads.
  wait_vmcnt<0>();

  RowOffsets<D> ro;
  ro.init(n, G);
  TrOffsets<D> to;
  to.init(lane);

  // Copy lanes: instruction i of a tile moves key rows RPI*i .. RPI*i+RPI-1;
  // this lane moves 16 bytes of row RPI*i + lrow into tile position (row,
  // lane % CPR), i.e. global chunk (lane % CPR) ^ swz(row).
  const int lrow = lane / CPR;
  int coff[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) coff[i] = ((lane % CPR) ^ swz<D>(RPI * i + lrow)) * 8;
  const int64_t row_el = (int64_t)Hkv * D;            // elements between consecutive tokens of a page

  // Pages of a tile's copy instructions, read one tile ahead of the copies
  // (their scalar-load latency then never delays a copy issue).
  struct TilePages {
    int id[NI];
  };
  auto tile_pages = [&](int tile) __attribute__((always_inline)) {
    TilePages tp;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int k0 = tile * kDecTile + RPI * i;
      tp.id[i] = k0 < kv_len ? load_const(p.page_ids, rq.page0 + k0 / P) : 0;
    }
    return tp;
  };
  auto issue_tile = [&](int tile, const TilePages &tp, int stage) __attribute__((always_inline)) {
    char *kd = wbase + (2 * stage) * TB;
    char *vd = kd + TB;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int k0 = tile * kDecTile + RPI * i;       // first key of the instruction (uniform)
      BufRsrc rk = make_rsrc(p.k_pages, 0), rv = make_rsrc(p.v_pages, 0);
      int voff = 0;
      if (k0 < kv_len) {
        const int pidx = k0 / P;
        const int page = tp.id[i];
        const int valid = min(P, kv_len - pidx * P);  // tokens held by this page
        const int64_t pbase = ((int64_t)page * P * Hkv + kvh) * D;
        const int bytes = (int)(((int64_t)(valid - 1) * row_el + D) * 2);
        rk = make_rsrc((const __bf16 *)p.k_pages + pbase, bytes);
        rv = make_rsrc((const __bf16 *)p.v_pages + pbase, bytes);
        voff = (int)(((int64_t)(k0 - pidx * P + lrow) * row_el + coff[i]) * 2);
      }
      dma16(rk, voff, kd + i * 1024);
      dma16(rv, voff, vd + i * 1024);
    }
  };

  float m_run = -INFINITY, l_run = 0.0f;
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = zero16();

  auto compute = [&](int tile, const char *kb, const char *vb) __attribute__((always_inline)) {
    const int key0 = tile * kDecTile;
    f32x16 s = zero16();
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) s = Mma<__bf16>::run(row_frag_at<D>(kb, ro, 0, st), qf[st], s);
    // Register j of lane group G holds key key0 + crow(j, G).
    if (key0 + kDecTile - 1 > kv_len - rq.n) {
      const int lim = my_lim - key0 - 4 * G;
#pragma unroll
      for (int j = 0; j < 16; ++j) s[j] = crow(j, 0) <= lim ? s[j] : -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[j]);
    mx = fmaxf(mx, xor32(mx)) * c;
    const float m_new = fmaxf(m_run, mx);
    const float mu = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = fast_exp2(m_run - mu);
    float ls = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      s[j] = fast_exp2(fmaf(s[j], c, -mu));
      ls += s[j];
    }
    l_run = l_run * alpha + ls;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bf16x8 pf = pack_bf16x8(s, h);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] = Mma<__bf16>::run(tr_frag_at<D>(vb, to, 16 * h, dt), pf, oacc[dt]);
    }
  };

  // Tiles tile0 + wave, + 4, ... ; the copy of the next one overlaps this one.
  int stage = 0;
  int t = w.tile0 + wave;
  TilePages next{};
  if (t < w.tile1) {
    issue_tile(t, tile_pages(t), 0);
    next = tile_pages(t + kDecWaves);
  }
  for (; t < w.tile1; t += kDecWaves) {
    const int tn = t + kDecWaves;
    if (tn < w.tile1) {
      issue_tile(tn, next, stage ^ 1);
      next = tile_pages(tn + kDecWaves);
      wait_vmcnt<2 * NI>();
    } else {
      wait_vmcnt<0>();
    }
    const char *kb = wbase + (2 * stage) * TB;
    compute(t, kb, kb + TB);
    stage ^= 1;
  }

  // Combine the four waves' partial softmax states (each wave has waited for
  // all of its copies). Per wave: O^T [dt][j][lane], then m and l per lane.
  __syncthreads();
  constexpr int XS = DT * 16 * 64 + 128;              // floats per wave
  float *x = reinterpret_cast<float *>(smem);
  float *mine = x + wave * XS;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) mine[(dt * 16 + j) * 64 + lane] = oacc[dt][j];
  mine[DT * 16 * 64 + lane] = m_run;
  mine[DT * 16 * 64 + 64 + lane] = l_run + xor32(l_run);
  __syncthreads();
  if (wave >= DT || !row_ok) return;
  const int dt = wave;
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < kDecWaves; ++v) M = fmaxf(M, x[v * XS + DT * 16 * 64 + lane]);
  float wv[kDecWaves];
  float L = 0.0f;
#pragma unroll
  for (int v = 0; v < kDecWaves; ++v) {
    const float mv = x[v * XS + DT * 16 * 64 + lane];
    wv[v] = (M == -INFINITY || mv == -INFINITY) ? 0.0f : fast_exp2(mv - M);
    L += wv[v] * x[v * XS + DT * 16 * 64 + 64 + lane];
  }
  f32x16 o = zero16();
#pragma unroll
  for (int v = 0; v < kDecWaves; ++v)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[j] += wv[v] * x[v * XS + (dt * 16 + j) * 64 + lane];
  const int64_t R = (int64_t)(rq.q0 + my_i) * Hq + my_h;   // row of q, o and the partial planes
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  const float lse = L > 0.0f ? (M + log2f(L)) * kLn2 : -INFINITY;
  if (w.split < 0) {
    __bf16 *op = (__bf16 *)p.o + R * D + dt * 32;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      store4(op + jj * 8 + G * 4, o[jj * 4] * inv, o[jj * 4 + 1] * inv, o[jj * 4 + 2] * inv, o[jj * 4 + 3] * inv);
    if (dt == 0 && G == 0 && p.lse != nullptr) p.lse[(int64_t)my_h * p.Tq + rq.q0 + my_i] = lse;
  } else {
    float *op = p.part_o + (w.split * p.plane + R) * D + dt * 32;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      store4(op + jj * 8 + G * 4, o[jj * 4] * inv, o[jj * 4 + 1] * inv, o[jj * 4 + 2] * inv, o[jj * 4 + 3] * inv);
    if (dt == 0 && G == 0) p.part_lse[w.split * p.plane + R] = lse;
  }
}

// LSE-weighted combination of a split request's partials: one thread per 4
// channels of a (query token, head) row.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeParams p) {
  constexpr int CPR = D / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t R = idx / CPR;
  const int c4 = (int)(idx % CPR);
  if (R >= p.plane) return;
  const int Hq = p.Hkv * p.g;
  const int t = (int)(R / Hq), h = (int)(R % Hq);
  const int ns = p.reqs[p.tok_req[t]].nsplit;
  if (ns <= 1) return;
  float mx = -INFINITY;
  for (int s = 0; s < ns; ++s) mx = fmaxf(mx, p.part_lse[s * p.plane + R]);
  float w_sum = 0.0f;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int s = 0; s < ns; ++s) {
    const float ls = p.part_lse[s * p.plane + R];
    const float wgt = ls == -INFINITY ? 0.0f : expf(ls - mx);
    w_sum += wgt;
    acc += wgt * *reinterpret_cast<const f32x4 *>(p.part_o + (s * p.plane + R) * D + c4 * 4);
  }
  const float inv = 1.0f / w_sum;
  store4((__bf16 *)p.o + R * D + c4 * 4, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  if (c4 == 0 && p.lse != nullptr) p.lse[(int64_t)h * p.Tq + t] = mx + logf(w_sum);
}

}  // namespace

hipError_t launch_decode_bf16(const DecodeParams &p, int D, int n_work, hipStream_t s) {
  if (D == 64)
    hipLaunchKernelGGL(decode_bf16_kernel<64>, dim3((unsigned)n_work), dim3(kDecWaves * 64), 0, s, p);
  else
    hipLaunchKernelGGL(decode_bf16_kernel<128>, dim3((unsigned)n_work), dim3(kDecWaves * 64), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_decode_merge_bf16(const DecodeParams &p, int D, hipStream_t s) {
  const int64_t n = p.plane * (D / 4);
  const unsigned grid = (unsigned)((n + 255) / 256);
  if (D == 64)
    hipLaunchKernelGGL(decode_merge_kernel<64>, dim3(grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(decode_merge_kernel<128>, dim3(grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace cas
