// Short-query / decode attention over a paged KV pool (forward only): the
// retrieved cartridges' pages, then the request's own pages, with the last
// n queries of the key sequence as the new tokens (paper: Section
// "Inference", paragraph "Cartridge RAG", and the appendix on cartridge
// sizes for the 16-token pages of the serving engine's KV cache).
//
// A decode step has very few query rows per (request, KV head) (n * g, e.g.
// 4) against thousands of keys, so the work is streaming K and V out of HBM.
// One workgroup takes a block of up to 16 packed rows of one (request, KV
// head) and a range of 32-key tiles (the host splits a request's key axis
// so that every compute unit holds two workgroups; partials are merged by
// their LSE). Its four waves work independently on every fourth tile of the
// range, so no wave ever waits on another until the end, where the four
// partial softmax states are combined through LDS. The products use
// v_mfma_f32_16x16x32_bf16, whose 16 columns fit the few rows of a decode
// step. K and V go from memory straight into registers, one tile ahead of
// their use: K already in the MFMA operand layout (each lane loads 16 bytes
// of one key row per step), V in whole rows, written into the wave's LDS
// tile just before its transposed reads for the PV product. Page addresses
// come from the page table (scalar loads, a tile ahead of the loads that
// use them). Per tile and wave: S^T = K Q^T, an online-softmax update, and
// O^T += V^T P^T with P^T straight from the score registers.
#include "cas_device.h"

namespace cas {

namespace {

constexpr int kDecWaves = 4;

typedef __attribute__((address_space(3))) char lds_char_t;

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int D>
__global__ __launch_bounds__(kDecWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_bf16_kernel(DecodeParams p) {
  static_assert(kDecRows == 16, "one 16-column MFMA block of rows");
  constexpr int NQ = D / 32;                  // 32-channel steps of the score product
  constexpr int NDB = D / 16;                 // 16-channel blocks of the PV product
  constexpr int TB = kDecTile * D * 2;        // bytes of one 32-key V tile
  constexpr int CPR = D / 8;                  // 16-byte chunks per key row
  constexpr int RPI = 64 / CPR;               // key rows per V load instruction
  constexpr int NI = kDecTile / RPI;          // V load instructions per tile
  constexpr int OS = NDB * 4 * 64;            // floats of one wave's O^T in the closing combine
  static_assert(OS * 4 == TB, "a wave's O^T fills its V tile");
  // Each wave's V tile (the closing combine reuses it for the wave's O^T);
  // m and l of every wave.
  __shared__ __attribute__((aligned(1024))) char vs[kDecWaves * TB];
  __shared__ __attribute__((aligned(16))) float ml[kDecWaves * 128];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15, bq = lane >> 4;    // MFMA column (row of the block) and k-group
  const DevDecodeWork w = load_const(p.work, (int)blockIdx.x);
  const DevDecodeReq rq = load_const(p.reqs, w.b);
  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g, P = p.page_size;
  const int kvh = __builtin_amdgcn_readfirstlane(w.kvh);
  const int kv_len = __builtin_amdgcn_readfirstlane(rq.kv_len);
  const int nrows = rq.n * g;
  const int my_row = w.row0 + j;
  const bool row_ok = my_row < nrows;
  const int my_i = my_row / g;                            // query index within the request
  const int my_h = kvh * g + (my_row - my_i * g);
  // Last key this row sees (rows past the block's end see every key: their
  // Q is zero and nothing of theirs is stored).
  const int my_lim = row_ok ? kv_len - rq.n + my_i : kv_len - 1;
  const float c = p.scale_log2;
  char *const vt = vs + wave * TB;

  // Q as the B operand: step st of lane (j, bq) is channels 32 st + 8 bq ..
  // + 7 of row j.
  bf16x8 qf[NQ];
  {
    const __bf16 *qp = (const __bf16 *)p.q + ((int64_t)(rq.q0 + (row_ok ? my_i : 0)) * Hq + my_h) * D + 8 * bq;
#pragma unroll
    for (int st = 0; st < NQ; ++st)
      qf[st] = row_ok ? *reinterpret_cast<const bf16x8 *>(qp + 32 * st) : Mma<__bf16>::zero();
  }

  // The pages of a tile's keys 0..15 (a) and 16..31 (b): one page when pages
  // hold 32 or more tokens, since tiles start at multiples of 32.
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
  // Element offset of key k0 + r (r < 32) of a tile in the pool; keys past
  // kv_len stand in for the tile's first key.
  auto key_off = [&](int k0, int r, const TilePages &tp) __attribute__((always_inline)) {
    const int rr = k0 + r < kv_len ? r : 0;
    const int page = rr < 16 ? tp.a : tp.b;
    return (((int64_t)page * P + ((k0 + rr) & (P - 1))) * Hkv + kvh) * D;
  };
  // K of a tile as the A operand: fragment kb * NQ + st of lane (j, bq) is
  // channels 32 st + 8 bq .. + 7 of key 16 kb + j.
  auto load_k = [&](int tile, const TilePages &tp, bf16x8 (&kr)[2 * NQ]) __attribute__((always_inline)) {
    const int k0 = tile * kDecTile;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const __bf16 *src = (const __bf16 *)p.k_pages + key_off(k0, 16 * kb + j, tp) + 8 * bq;
#pragma unroll
      for (int st = 0; st < NQ; ++st) kr[kb * NQ + st] = *reinterpret_cast<const bf16x8 *>(src + 32 * st);
    }
  };
  // V of a tile in whole rows: load i of a lane is chunk lane % CPR of key
  // row RPI * i + lane / CPR.
  auto load_v = [&](int tile, const TilePages &tp, bf16x8 (&vr)[NI]) __attribute__((always_inline)) {
    const int k0 = tile * kDecTile;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const __bf16 *src = (const __bf16 *)p.v_pages + key_off(k0, RPI * i + lane / CPR, tp) + (lane % CPR) * 8;
      vr[i] = *reinterpret_cast<const bf16x8 *>(src);
    }
  };
  // V rows into the wave's LDS tile (16-byte chunks XOR-swizzled by row);
  // rows past kv_len are written as zeros.
  auto write_v = [&](int tile, const bf16x8 (&vr)[NI]) __attribute__((always_inline)) {
    const int k0 = tile * kDecTile;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = RPI * i + lane / CPR;
      const bf16x8 v = k0 + r < kv_len ? vr[i] : Mma<__bf16>::zero();
      *reinterpret_cast<bf16x8 *>(vt + r * (D * 2) + (((lane % CPR) ^ swz<D>(r)) << 4)) = v;
    }
  };
  // V^T as the A operand of the PV product for channel block db: lane (j, bq)
  // holds channel 16 db + j of keys 4 bq .. 4 bq + 3 and 16 + 4 bq .. + 3, the
  // keys its P^T registers hold. Each transposed read of a 16-lane group
  // covers 4 key rows x 16 channels; lane j addresses row j / 4, channels
  // 4 (j % 4) .. + 3 of it and receives channel j of all four rows.
  auto vt_frag = [&](int db) __attribute__((always_inline)) {
    const lds_char_t *base = (const lds_char_t *)vt;
    i16x4 part[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int row = 16 * h + 4 * bq + (j >> 2);
      const int col = 16 * db + 4 * (j & 3);
      const int off = row * (D * 2) + (((col >> 3) ^ swz<D>(row)) << 4) + ((col >> 2) & 1) * 8;
      part[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(base + off));
    }
    typedef short i16x8 __attribute__((ext_vector_type(8)));
    return __builtin_bit_cast(bf16x8, (i16x8)__builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
  };

  float m_run = -INFINITY, l_run = 0.0f;
  f32x4 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto compute = [&](int tile, const bf16x8 (&kr)[2 * NQ]) __attribute__((always_inline)) {
    const int key0 = tile * kDecTile;
    // S^T: register e of score block kb of lane (j, bq) is key 16 kb + 4 bq + e, row j.
    f32x4 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int st = 0; st < NQ; ++st) s[kb] = mfma16(kr[kb * NQ + st], qf[st], s[kb]);
    }
    if (key0 + kDecTile - 1 > kv_len - rq.n) {
      const int lim = my_lim - key0 - 4 * bq;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) s[kb][e] = 16 * kb + e <= lim ? s[kb][e] : -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, s[kb][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c;
    const float m_new = fmaxf(m_run, mx);
    const float mu = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = fast_exp2(m_run - mu);
    float ls = 0.0f;
    bf16x8 pf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float pv = fast_exp2(fmaf(s[kb][e], c, -mu));
        ls += pv;
        pf[4 * kb + e] = (__bf16)pv;
      }
    l_run = l_run * alpha + ls;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      oacc[db] *= alpha;
      oacc[db] = mfma16(vt_frag(db), pf, oacc[db]);
    }
  };

  // Tiles tile0 + wave, + 4, ...: the K and V loads of the wave's next tile
  // go out before this tile's V is written to LDS and its products run;
  // the page ids come one tile earlier still.
  bf16x8 kra[2 * NQ], krb[2 * NQ], vra[NI], vrb[NI];
  int t = w.tile0 + wave;
  TilePages next{};
  if (t < w.tile1) {
    const TilePages tp = tile_pages(t);
    load_k(t, tp, kra);
    load_v(t, tp, vra);
    next = tile_pages(t + kDecWaves);
  }
  auto step = [&](int tile, bf16x8 (&kc)[2 * NQ], bf16x8 (&vc)[NI], bf16x8 (&kn)[2 * NQ], bf16x8 (&vn)[NI])
                  __attribute__((always_inline)) {
    const int tn = tile + kDecWaves;
    if (tn < w.tile1) {
      const TilePages pn = next;
      load_k(tn, pn, kn);
      load_v(tn, pn, vn);
      next = tile_pages(tn + kDecWaves);
    }
    write_v(tile, vc);
    compute(tile, kc);
  };
  for (; t < w.tile1; t += 2 * kDecWaves) {
    step(t, kra, vra, krb, vrb);
    if (t + kDecWaves >= w.tile1) break;
    step(t + kDecWaves, krb, vrb, kra, vra);
  }

  // Combine the four waves' partial softmax states. Per wave: O^T
  // [db][e][lane] in its V tile, m and the row sum of l per lane in ml.
  const float l_row = l_run + __shfl_xor(l_run, 16, 64);
  const float l_all = l_row + __shfl_xor(l_row, 32, 64);
  __syncthreads();   // every wave is done with its V tile
  float *const mine = reinterpret_cast<float *>(vt);
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int e = 0; e < 4; ++e) mine[(db * 4 + e) * 64 + lane] = oacc[db][e];
  ml[wave * 128 + lane] = m_run;
  ml[wave * 128 + 64 + lane] = l_all;
  __syncthreads();
  if (!row_ok) return;
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
  const int64_t R = (int64_t)(rq.q0 + my_i) * Hq + my_h;   // row of q, o and the partial planes
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  // Wave v stores channel blocks v, v + 4, ...: lane (j, bq) channels
  // 16 db + 4 bq .. + 3 of row j.
  for (int db = wave; db < NDB; db += kDecWaves) {
    f32x4 o = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int v = 0; v < kDecWaves; ++v) {
      const float *ov = reinterpret_cast<const float *>(vs + v * TB);
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] += wv[v] * ov[(db * 4 + e) * 64 + lane];
    }
    const int ch = 16 * db + 4 * bq;
    if (w.split < 0)
      store4((__bf16 *)p.o + R * D + ch, o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
    else
      store4(p.part_o + (w.split * p.plane + R) * D + ch, o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
  }
  if (wave == 0 && bq == 0) {
    const float lse = L > 0.0f ? (M + log2f(L)) * kLn2 : -INFINITY;
    if (w.split < 0) {
      if (p.lse != nullptr) p.lse[(int64_t)my_h * p.Tq + rq.q0 + my_i] = lse;
    } else {
      p.part_lse[w.split * p.plane + R] = lse;
    }
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
