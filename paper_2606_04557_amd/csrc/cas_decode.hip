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
// so that every compute unit holds two workgroups; partials are merged by
// their LSE). Its four waves work independently on every fourth tile of the
// range, so no wave ever waits on another until the end, where the four
// partial softmax states are combined through LDS. K goes straight from
// memory into the MFMA operand registers (each lane loads 16 bytes of one
// key row per step); V goes through two LDS stages per wave, filled by
// direct buffer->LDS copies, for the transposed reads of the PV product.
// The two stages are separate LDS objects and the loop alternates them at
// compile time, so the compiler can tell a stage's transposed reads from
// the copies into the other one and does not wait for those copies.
// Page addresses come from the page table (one scalar load per page, a tile
// ahead). Per tile and wave: S^T = K Q^T (MFMA, K and Q in registers), an
// online-softmax update, and O^T += V^T P^T (MFMA, V^T by transposed LDS
// reads, P straight from the score registers).
#include "cas_device.h"

namespace cas {

namespace {

constexpr int kDecWaves = 4;

template <int D>
__global__ __launch_bounds__(kDecWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_bf16_kernel(DecodeParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int TB = kDecTile * D * 2;        // bytes of one 32-key V tile
  constexpr int CPR = D / 8;                  // 16-byte chunks per key row
  constexpr int RPI = 64 / CPR;               // key rows per copy instruction
  constexpr int NI = kDecTile / RPI;          // copy instructions per V tile
  constexpr int OS = DT * 16 * 64;            // floats of one wave's O^T in the closing combine
  static_assert(kDecTile % RPI == 0 && 16 % RPI == 0, "copy instructions stay within a page");
  static_assert(2 * OS * 4 == kDecWaves * TB, "two waves' O^T fill one stage object");
  static_assert(2 * (2 * kDecWaves * TB + kDecWaves * 128 * 4) <= 160 * 1024, "two workgroups per compute unit");
  // V stages 0 and 1 of every wave; the closing combine puts the O^T of
  // waves 0-1 into the first and of waves 2-3 into the second, m and l into ml.
  __shared__ __attribute__((aligned(1024))) char vs0[kDecWaves * TB];
  __shared__ __attribute__((aligned(1024))) char vs1[kDecWaves * TB];
  __shared__ __attribute__((aligned(16))) float ml[kDecWaves * 128];

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
  char *const st0 = vs0 + wave * TB;
  char *const st1 = vs1 + wave * TB;

  bf16x8 qf[NSTEP];
  if (row_ok) {
    const __bf16 *qp = (const __bf16 *)p.q + ((int64_t)(rq.q0 + my_i) * Hq + my_h) * D;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) qf[st] = *reinterpret_cast<const bf16x8 *>(qp + st * 16 + G * 8);
  } else {
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) qf[st] = Mma<__bf16>::zero();
  }
  // No wait here: these loads are older than every tile load, so the first
  // tile's partial wait covers them, and their latency overlaps the first
  // tile's.

  TrOffsets<D> to;
  to.init(lane);

  // Copy lanes: instruction i of a V tile moves key rows RPI*i .. RPI*i+RPI-1;
  // this lane moves 16 bytes of row RPI*i + lrow into tile position (row,
  // lane % CPR), i.e. global chunk (lane % CPR) ^ swz(row).
  const int lrow = lane / CPR;
  int coff[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) coff[i] = ((lane % CPR) ^ swz<D>(RPI * i + lrow)) * 8;
  const int64_t row_el = (int64_t)Hkv * D;            // elements between consecutive tokens of a page

  // The pages of a tile's keys 0..15 (a) and 16..31 (b): one page when pages
  // hold 32 or more tokens, since tiles start at multiples of 32. Read one
  // tile ahead of their loads, so the scalar-load latency never delays one.
  struct TilePages {
    int a, b;
  };
  auto tile_pages = [&](int tile) __attribute__((always_inline)) {
    TilePages tp{0, 0};
    const int k0 = tile * kDecTile;
    if (k0 < kv_len) {
      tp.a = load_const(p.page_ids, rq.page0 + k0 / P);
      tp.b = k0 + 16 < kv_len ? load_const(p.page_ids, rq.page0 + (k0 + 16) / P) : tp.a;
    }
    return tp;
  };
  // K of a tile into the MFMA A-operand registers: step st of lane (n, G)
  // is channels 16 st + 8 G .. + 7 of the tile's key n. Keys past kv_len
  // load the tile's first key instead; their scores are masked.
  auto load_k = [&](int tile, const TilePages &tp, bf16x8 (&kr)[NSTEP]) __attribute__((always_inline)) {
    const int k0 = tile * kDecTile;
    const int kk = k0 + n < kv_len ? n : 0;
    const int page = kk < 16 ? tp.a : tp.b;
    const int tok = (k0 + kk) & (P - 1);
    const __bf16 *src = (const __bf16 *)p.k_pages + (((int64_t)page * P + tok) * Hkv + kvh) * D + 8 * G;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) kr[st] = *reinterpret_cast<const bf16x8 *>(src + 16 * st);
  };
  // V of a tile into the wave's stage vd; rows past kv_len, and every row
  // when the tile is not live, read as zero.
  auto issue_v = [&](int tile, const TilePages &tp, char *vd, bool live) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int k0 = tile * kDecTile + RPI * i;       // first key of the instruction (uniform)
      BufRsrc rv = make_rsrc(p.v_pages, 0);
      int voff = 0;
      if (live && k0 < kv_len) {
        const int pidx = k0 / P;
        const int page = RPI * i < 16 ? tp.a : tp.b;
        const int valid = min(P, kv_len - pidx * P);  // tokens held by this page
        const int64_t pbase = ((int64_t)page * P * Hkv + kvh) * D;
        const int bytes = (int)(((int64_t)(valid - 1) * row_el + D) * 2);
        rv = make_rsrc((const __bf16 *)p.v_pages + pbase, bytes);
        voff = (int)(((int64_t)(k0 - pidx * P + lrow) * row_el + coff[i]) * 2);
      }
      dma16(rv, voff, vd + i * 1024);
    }
  };

  float m_run = -INFINITY, l_run = 0.0f;
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = zero16();

  // S^T of a tile from K in registers; K of the wave's next tile (pages
  // nk) is then loaded into the same registers, so its latency hides behind
  // this tile's softmax and PV product.
  bf16x8 kr[NSTEP];
  auto compute = [&](int tile, const char *vb, int tnext, const TilePages &nk) __attribute__((always_inline)) {
    const int key0 = tile * kDecTile;
    f32x16 s = zero16();
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) s = Mma<__bf16>::run(kr[st], qf[st], s);
    if (tnext < w.tile1) load_k(tnext, nk, kr);
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

  // Tiles tile0 + wave, + 4, ..., alternately from stage 0 and stage 1.
  // Outstanding loads, oldest first, when a tile's wait comes: its V copies
  // (issued an iteration earlier), its K (issued during the previous tile's
  // softmax), then the next tile's V copies (issued just before the wait),
  // which alone may stay in flight. After the wave's last tile the next
  // copies still go out, reading nothing and writing zeros: with the copy
  // and the wait unconditional the compiler keeps the partial count instead
  // of waiting for every copy before the transposed reads.
  int t = w.tile0 + wave;
  TilePages next{};
  if (t < w.tile1) {
    const TilePages tp = tile_pages(t);
    load_k(t, tp, kr);
    issue_v(t, tp, st0, true);
    next = tile_pages(t + kDecWaves);
  }
  auto step = [&](int tile, const char *cur, char *other) __attribute__((always_inline)) {
    const int tn = tile + kDecWaves;
    const TilePages pn = next;
    issue_v(tn, pn, other, tn < w.tile1);
    next = tile_pages(tn + kDecWaves);
    wait_vmcnt<NI>();
    compute(tile, cur, tn, pn);
  };
  for (; t < w.tile1; t += 2 * kDecWaves) {
    step(t, st0, st1);
    if (t + kDecWaves >= w.tile1) break;
    step(t + kDecWaves, st1, st0);
  }
  wait_vmcnt<0>();   // the closing copies land before the combine reuses the stages

  // Combine the four waves' partial softmax states (each wave has waited for
  // all of its copies). Per wave: O^T [dt][j][lane], and m and l per lane.
  __syncthreads();
  auto obuf = [&](int v) __attribute__((always_inline)) {
    return reinterpret_cast<float *>(v < 2 ? vs0 : vs1) + (v & 1) * OS;
  };
  float *mine = obuf(wave);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) mine[(dt * 16 + j) * 64 + lane] = oacc[dt][j];
  ml[wave * 128 + lane] = m_run;
  ml[wave * 128 + 64 + lane] = l_run + xor32(l_run);
  __syncthreads();
  if (wave >= DT || !row_ok) return;
  const int dt = wave;
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < kDecWaves; ++v) M = fmaxf(M, ml[v * 128 + lane]);
  float wv[kDecWaves];
  float L = 0.0f;
#pragma unroll
  for (int v = 0; v < kDecWaves; ++v) {
    const float mv = ml[v * 128 + lane];
    wv[v] = (M == -INFINITY || mv == -INFINITY) ? 0.0f : fast_exp2(mv - M);
    L += wv[v] * ml[v * 128 + 64 + lane];
  }
  f32x16 o = zero16();
#pragma unroll
  for (int v = 0; v < kDecWaves; ++v)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[j] += wv[v] * obuf(v)[(dt * 16 + j) * 64 + lane];
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
