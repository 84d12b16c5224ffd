// bf16 fast path of multi-cartridge prefix attention for gfx950.
//
// All three kernels use 512-thread workgroups (8 waves, two per SIMD, so one
// wave's softmax VALU work overlaps the other's MFMA work), swizzled row tiles
// in LDS filled by asynchronous direct global->LDS copies, double buffering
// (the copy of tile i+1 is in flight while tile i is computed; one barrier per
// tile), and ds_read_b64_tr_b16 for every operand that is reduced along its
// row axis (V in the forward, K in dQ, Q and dO in dK/dV).
#include <type_traits>
#include <utility>

#include "cas_device.h"

namespace cas {

namespace {

constexpr int kNW = 8;                 // waves per workgroup
constexpr int kFastThreads = kNW * 64;
constexpr int kKT = 64;                // keys per tile (forward, dQ)
constexpr int kFastRowsPerWave = 32;
constexpr int kFastRowsPerWg = kNW * kFastRowsPerWave;   // 256
constexpr float kRefMargin = 64.0f;    // forward: largest score above the row's fixed offset (log2 units)

struct TileInfo {
  const __bf16 *kp;
  const __bf16 *vp;
  int st;      // token stride in elements (the host keeps 128 rows within 32-bit offsets)
  int nvalid;
  int self0;   // first self key of the tile, or -1 for a cartridge tile
};

// f(integral_constant<int, 0>) ... f(integral_constant<int, N-1>), unrolled.
template <typename F, int... Ks>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, Ks...>) {
  (f(std::integral_constant<int, Ks>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Scheduling groups: the next n MFMAs / LDS reads of the region, in order.
template <int N>
__device__ __forceinline__ void sched_mfma() { __builtin_amdgcn_sched_group_barrier(0x008, N, 0); }
template <int N>
__device__ __forceinline__ void sched_ds_read() { __builtin_amdgcn_sched_group_barrier(0x100, N, 0); }

struct TileMask {
  int nvalid;
  int self0;
};

// Per-lane share of the direct-to-LDS copies of an R-row tile: the tile row
// and element offset (swizzle applied) of each 16-byte chunk this lane moves
// are fixed for the whole kernel, so a tile copy costs one multiply-add and
// one copy instruction per chunk.
template <int D, int R, int NW>
struct CopyLanes {
  static constexpr int CPR = D / 8;
  static constexpr int NI = R * CPR / 64;             // 1 KiB wave instructions per tile
  static constexpr int PER = (NI + NW - 1) / NW;      // instructions per wave
  int row[PER];
  int coff[PER];
  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int pos = (wave + i * NW) * 64 + lane;
      const int r = pos / CPR;
      row[i] = r;
      coff[i] = ((pos % CPR) ^ swz<D>(r)) * 8;
    }
  }
  // Rows at or beyond nvalid (>= 1) re-read row nvalid-1 (finite; masked
  // later). The copies go through a buffer resource spanning exactly the
  // tile's rows (an out-of-range offset would read zeros, not fault), and
  // as MUBUF LDS loads they are counted on vmcnt alone.
  __device__ __forceinline__ void issue(char *tile, const __bf16 *base, int st, int nvalid, int wave) const {
    const BufRsrc rs = make_rsrc(base, ((nvalid - 1) * st + D) * 2);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int inst = wave + i * NW;
      if (NI % NW == 0 || inst < NI) dma16(rs, (min(row[i], nvalid - 1) * st + coff[i]) * 2, tile + inst * 1024);
    }
  }
};

// Workgroup barrier that orders LDS use: this wave's LDS reads have returned,
// and the compiler moves no memory access across it. Outstanding direct
// global->LDS copies are not waited for (wait_vmcnt does that).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt, expcnt untouched
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Key tiles of one batch row at one KV head, from the row's slice of the
// host-built tile table (one scalar load per tile): the prefix tiles in
// segment order, then the causal self tiles.
struct TileTable {
  const DevTile *tiles;
  int tile_begin;   // row's first table entry
  int ptiles;       // prefix tiles of the row
  int kvh;

  __device__ __forceinline__ void init(const DevTile *t, const DevRow &row, int kvh_) {
    tiles = t;
    tile_begin = __builtin_amdgcn_readfirstlane(row.tile_begin);
    ptiles = __builtin_amdgcn_readfirstlane(row.prefix_tiles);
    kvh = kvh_;
  }
  __device__ __forceinline__ int nvalid(int tile) const {
    return load_const(&tiles[__builtin_amdgcn_readfirstlane(tile_begin + tile)].nvalid, 0);
  }
  __device__ __forceinline__ TileInfo at(int tile) const {
    const DevTile t = load_const(tiles, __builtin_amdgcn_readfirstlane(tile_begin + tile));
    const int64_t hoff = kvh * t.stride_head;
    TileInfo ti;
    ti.kp = (const __bf16 *)t.k + hoff;
    ti.vp = (const __bf16 *)t.v + hoff;
    ti.st = t.stride_tok;
    ti.nvalid = t.nvalid;
    ti.self0 = tile < ptiles ? -1 : (tile - ptiles) * kKT;
    return ti;
  }
};

}  // namespace

// ---------------------------------------------------------------------------
// Forward: ping-pong between the two waves of each SIMD.
//
// Waves 0-3 (group A) and 4-7 (group B) occupy one slot on each of the four
// SIMDs. Per key tile i a wave runs a matrix phase G_i (O += V_{i-1}^T P_{i-1}
// and S_i = K_i Q^T: 32 MFMAs in one scheduling region) and a softmax phase
// X_i (mask, row max, exp2, row sums, bf16 packing of P_i: VALU only). Group B
// runs one phase behind group A and every phase ends in a workgroup barrier,
// so on each SIMD one wave's MFMA stream runs beside the other wave's softmax.
//
// LDS: three K and three V tile buffers. Only group B copies: at the start of
// phase 2i (while it runs a softmax phase) it issues K_{i+2} and V_{i+1} into
// the buffers that K_{i-1} and V_{i-2} left free after phase 2i-1, and at the
// end of phase 2i it waits for the copies it issued at phase 2i-2, which
// group A's G_{i+1} reads at phase 2i+2.
//
// Softmax reference: a row's exponent offset m is fixed by the first tile in
// which it sees a key, and never moved, so O is never rescaled in the loop.
// Later scores may exceed m by up to kRefMargin (log2 units) -- P stays below
// 2^kRefMargin, far inside fp32 and bf16 range. A row that goes beyond the
// margin flags its workgroup; it records every row's exact maximum, and a
// second launch (FIXUP) recomputes only the flagged workgroups with m set to
// that maximum. Unflagged workgroups of the second launch exit at once.
// ---------------------------------------------------------------------------
template <int D, bool FIXUP>
__global__ __launch_bounds__(kFastThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void fwd_bf16_kernel(FwdParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int TB = kKT * D * 2;
  __shared__ __attribute__((aligned(1024))) char kb0[TB];
  __shared__ __attribute__((aligned(1024))) char kb1[TB];
  __shared__ __attribute__((aligned(1024))) char kb2[TB];
  __shared__ __attribute__((aligned(1024))) char vb0[TB];
  __shared__ __attribute__((aligned(1024))) char vb1[TB];
  __shared__ __attribute__((aligned(1024))) char vb2[TB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int G = lane >> 5, n = lane & 31;
  int bid = blockIdx.x;
  const int qblk = __builtin_amdgcn_readfirstlane(bid % p.nqblk);
  bid /= p.nqblk;
  const int kvh = __builtin_amdgcn_readfirstlane(bid % p.Hkv);
  bid /= p.Hkv;
  const int split = __builtin_amdgcn_readfirstlane(bid % p.splits);
  const int b = __builtin_amdgcn_readfirstlane(bid / p.splits);
  if constexpr (FIXUP) {
    if (load_const(p.ovf_flag, (int)blockIdx.x) == 0) return;
  }

  const int g = p.g, Sq = p.Sq, Hkv = p.Hkv, Hq = Hkv * g, nrows = p.nrows;
  const int wg_row0 = qblk * kFastRowsPerWg;
  const int wg_row1 = min(nrows, wg_row0 + kFastRowsPerWg);
  const int row0 = wg_row0 + wave * kFastRowsPerWave;
  const bool wave_active = row0 < nrows;
  const int wave_t_lo = row0 / g;
  const int wave_t_hi = (min(row0 + kFastRowsPerWave, nrows) - 1) / g;
  const int wg_t_hi = (wg_row1 - 1) / g;
  const int my_row = row0 + n;
  const int my_t = my_row / g;
  const float c = p.scale_log2;
  // This row's slot in the per-split row-maximum buffer.
  const int64_t mrow = (((int64_t)split * p.B + b) * Hkv + kvh) * nrows + min(my_row, nrows - 1);

  // Wave-uniform tile range of this split (readfirstlane keeps it, and every
  // tile-table read that depends on it, in scalar registers).
  const DevRow row = load_const(p.rows, b);
  const int ptiles = __builtin_amdgcn_readfirstlane(row.prefix_tiles);
  const int ntiles = ptiles + wg_t_hi / kKT + 1;
  const int tb = __builtin_amdgcn_readfirstlane((int)((int64_t)ntiles * split / p.splits));
  const int te = __builtin_amdgcn_readfirstlane((int)((int64_t)ntiles * (split + 1) / p.splits));
  const int nt = te - tb;
  TileTable tt;
  tt.init(p.tiles, row, kvh);

  RowOffsets<D> ro;
  ro.init(n, G);
  TrOffsets<D> to;
  to.init(lane);

  bf16x8 qf[NSTEP];
  if (my_row < nrows) {
    const __bf16 *rp = (const __bf16 *)p.q + (((int64_t)b * Sq + my_t) * Hq + kvh * g + (my_row - my_t * g)) * D;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) qf[st] = *reinterpret_cast<const bf16x8 *>(rp + st * 16 + G * 8);
  } else {
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) qf[st] = Mma<__bf16>::zero();
  }
  // Tile copies are waited for with partial vmcnt counts, which must not
  // include these loads.
  wait_vmcnt<0>();

  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = zero16();
  // Exponent offset of this lane's row: fixed by its first visible tile, or
  // (FIXUP) the exact row maximum the first launch recorded.
  float m_run = FIXUP ? p.row_max[mrow] : -INFINITY;
  float m_max = -INFINITY;    // exact running row max
  float l_run = 0.0f;
  bool beyond = false;        // a score exceeded m_run + kRefMargin

  // Group B's share of every tile copy (4 waves).
  CopyLanes<D, kKT, 4> cl;
  cl.init(wave & 3, lane);
  constexpr int kCopyInst = CopyLanes<D, kKT, 4>::PER;   // per wave per K or V tile

  // Scores of the tile between its G and X phases; P of the tile between its
  // X phase and the next G phase.
  f32x16 s0 = zero16(), s1 = zero16();
  bf16x8 pf[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int s = 0; s < 2; ++s) pf[a][s] = Mma<__bf16>::zero();

  // Local tile j: whether this wave sees any key of it (self tiles past the
  // wave's last query position are skipped), and its mask data.
  auto self0_of = [&](int j) __attribute__((always_inline)) {
    return tb + j < ptiles ? -1 : (tb + j - ptiles) * kKT;
  };
  auto live = [&](int j) __attribute__((always_inline)) {
    const int s0_ = self0_of(j);
    return wave_active && !(s0_ >= 0 && s0_ > wave_t_hi);
  };

  // Matrix phase as one software-pipelined sequence of MFMAs: the PV product
  // of the previous tile (16 MFMAs, two transposed LDS reads per fragment),
  // then the scores of this one (16 MFMAs, one LDS read per fragment). The
  // fragment of MFMA k+LEAD is read while MFMA k runs, into a ring of LEAD+1
  // registers, and the scheduling groups pin exactly that order, so the LDS
  // latency hides behind the MFMA pipe across the PV -> S boundary too.
  auto matrix = [&](auto DO_PV, auto DO_S, const char *kb, const char *vb) __attribute__((always_inline)) {
    constexpr bool PV = decltype(DO_PV)::value, S = decltype(DO_S)::value;
    constexpr int NPV = PV ? 4 * DT : 0;          // PV MFMAs
    constexpr int N = NPV + (S ? 2 * NSTEP : 0);  // all MFMAs
    constexpr int LEAD = 4, R = LEAD + 1;
    // MFMA k < NPV: s = k / (2*DT), dt = (k / 2) % DT, key half hh = k % 2.
    // MFMA k >= NPV: st = (k - NPV) / 2, score half hh = (k - NPV) % 2.
    auto load = [&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < NPV) {
        constexpr int s = k / (2 * DT), dt = (k / 2) % DT, hh = k % 2;
        return tr_frag_at<D>(vb, to, 32 * hh + 16 * s, dt);
      } else {
        constexpr int st = (k - NPV) / 2, hh = (k - NPV) % 2;
        return row_frag_at<D>(kb, ro, 32 * hh, st);
      }
    };
    auto mma = [&](auto K, const bf16x8 &f) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < NPV) {
        constexpr int s = k / (2 * DT), dt = (k / 2) % DT, hh = k % 2;
        oacc[dt] = Mma<__bf16>::run(f, pf[hh][s], oacc[dt]);
      } else {
        constexpr int st = (k - NPV) / 2, hh = (k - NPV) % 2;
        if constexpr (hh == 0) s0 = Mma<__bf16>::run(f, qf[st], s0);
        else s1 = Mma<__bf16>::run(f, qf[st], s1);
      }
    };
    if constexpr (S) {
      s0 = zero16();
      s1 = zero16();
    }
    bf16x8 ring[R];
    static_for<LEAD>([&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < N) ring[k % R] = load(K);
    });
    static_for<N>([&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k + LEAD < N) ring[(k + LEAD) % R] = load(std::integral_constant<int, k + LEAD>{});
      mma(K, ring[k % R]);
    });
    // Scheduling groups: the LEAD first fragments, then per MFMA k the reads
    // of fragment k+LEAD.
    static_for<LEAD>([&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < N) sched_ds_read<(k < NPV ? 2 : 1)>();
    });
    static_for<N>([&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      sched_mfma<1>();
      if constexpr (k + LEAD < N) sched_ds_read<(k + LEAD < NPV ? 2 : 1)>();
    });
  };
  auto softmax = [&](auto MASK, int lim) __attribute__((always_inline)) {
    if constexpr (decltype(MASK)::value) {
      // lim: last visible key of this lane's query within the tile. Register
      // j of group G holds key crow(j, G) = crow(j, 0) + 4G, so comparing
      // lim - 4G against compile-time constants needs no index registers.
      const int limg = lim - 4 * G;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        s0[j] = crow(j, 0) <= limg ? s0[j] : -INFINITY;
        s1[j] = 32 + crow(j, 0) <= limg ? s1[j] : -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 16; j += 2) mx = fmaxf(fmaxf(mx, fmaxf(s0[j], s1[j])), fmaxf(s0[j + 1], s1[j + 1]));
    const float mt = fmaxf(mx, xor32(mx)) * c;
    if constexpr (!FIXUP) {
      m_run = (m_run == -INFINITY) ? mt : m_run;
      beyond = beyond || (mt > m_run + kRefMargin);
      m_max = fmaxf(m_max, mt);
    }
    const float mu = (m_run == -INFINITY) ? 0.0f : m_run;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      s0[j] = fast_exp2(fmaf(s0[j], c, -mu));
      s1[j] = fast_exp2(fmaf(s1[j], c, -mu));
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      pf[0][s] = pack_bf16x8(s0, s);
      pf[1][s] = pack_bf16x8(s1, s);
    }
    // Row sums in fp32 (the LSE needs them to better than bf16 rounding).
    float la = 0.0f, lb = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      la += s0[j];
      lb += s1[j];
    }
    l_run += la + lb;
  };

  // G_j: PV of tile j-1 (V_{j-1} in vbp) and scores of tile j (K_j in kb),
  // always both: P is zero where there is no previous tile or it was not
  // visible, and scores of a tile past the end or not visible are never
  // read. (Conditionally skipping either half would make the register
  // allocator copy the accumulators around every such branch.)
  auto gphase = [&](int j, const char *kb, const char *vbp) __attribute__((always_inline)) {
    if (j <= nt && wave_active) matrix(std::true_type{}, std::true_type{}, kb, vbp);
  };
  auto xphase = [&](int j) __attribute__((always_inline)) {
    if (j < 0 || j >= nt) return;
    if (!live(j)) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int s = 0; s < 2; ++s) pf[a][s] = Mma<__bf16>::zero();
      return;
    }
    const int self0 = self0_of(j);
    const int nvalid = __builtin_amdgcn_readfirstlane(tt.nvalid(tb + j));
    if (nvalid < kKT || (self0 >= 0 && self0 + kKT - 1 > wave_t_lo)) {
      const int lim = self0 < 0 ? nvalid - 1 : min(nvalid - 1, my_t - self0);
      softmax(std::true_type{}, lim);
    } else {
      softmax(std::false_type{}, kKT - 1);
    }
  };

  // Group B's copies. tk: the K tile issued last (tile i+1 when phase 2i
  // starts), whose V is issued next.
  TileInfo tk;
  auto copy_k = [&](char *kbn, int j) __attribute__((always_inline)) {
    tk = tt.at(tb + j);
    cl.issue(kbn, tk.kp, tk.st, tk.nvalid, wave & 3);
  };
  // Phase 2i: K_{i+2} and V_{i+1}; then the copies of phase 2i-2 are waited for.
  auto issue = [&](int i, char *kbn, char *vbn) __attribute__((always_inline)) {
    if (i + 1 < nt) cl.issue(vbn, tk.vp, tk.st, tk.nvalid, wave & 3);
    if (i + 2 < nt) copy_k(kbn, i + 2);
  };
  auto wait_older = [&](int i) __attribute__((always_inline)) {
    // The newest batch (issued this phase) may still be in flight.
    if (i + 2 < nt) wait_vmcnt<2 * kCopyInst>();
    else if (i + 1 < nt) wait_vmcnt<kCopyInst>();
    else wait_vmcnt<0>();
  };

  if (nt > 0) {
    // G_0 multiplies V buffer 2 by P = 0: clear it so no stale bit pattern
    // (a NaN) can reach O.
    for (int i = tid; i < TB / 16; i += kFastThreads) reinterpret_cast<uint4 *>(vb2)[i] = uint4{0, 0, 0, 0};
    // Prologue (group B): K_0, then K_1 and V_0.
    if (grp == 1) {
      copy_k(kb0, 0);
      wait_vmcnt<0>();
      const TileInfo t0 = tk;
      cl.issue(vb0, t0.vp, t0.st, t0.nvalid, wave & 3);
      if (nt > 1) copy_k(kb1, 1);
    }
    lds_barrier();
    // Six phases per iteration (three tiles), so every buffer is a fixed LDS
    // address: G_i reads K_i from kb[i%3] and V_{i-1} from vb[(i-1)%3]; the
    // copies of phase 2i go to kb[(i+2)%3] and vb[(i+1)%3]. Each group runs
    // its own copy of the loop (straight-line phases); s_barrier pairs them.
    auto run = [&](auto GROUP_A) __attribute__((always_inline)) {
      constexpr bool A = decltype(GROUP_A)::value;
      auto even = [&](int i, const char *kbi, const char *vbp, char *kbn, char *vbn) __attribute__((always_inline)) {
        if constexpr (A) {
          gphase(i, kbi, vbp);
        } else {
          issue(i, kbn, vbn);
          xphase(i - 1);
          wait_older(i);
        }
        lds_barrier();
      };
      auto odd = [&](int i, const char *kbi, const char *vbp) __attribute__((always_inline)) {
        if constexpr (A) xphase(i);
        else gphase(i, kbi, vbp);
        lds_barrier();
      };
      for (int i = 0; i <= nt; i += 3) {
        even(i, kb0, vb2, kb2, vb1);
        odd(i, kb0, vb2);
        if (i + 1 > nt) break;
        even(i + 1, kb1, vb0, kb0, vb2);
        odd(i + 1, kb1, vb0);
        if (i + 2 > nt) break;
        even(i + 2, kb2, vb1, kb1, vb0);
        odd(i + 2, kb2, vb1);
      }
    };
    if (grp == 0) run(std::true_type{});
    else run(std::false_type{});
  }
  if constexpr (!FIXUP) {
    // Every wave reaches this point: flag the workgroup and keep the exact
    // row maxima if any row went beyond the margin.
    const int any = __syncthreads_or(beyond ? 1 : 0);
    if (tid == 0) p.ovf_flag[blockIdx.x] = any;
    if (any && my_row < nrows && G == 0) p.row_max[mrow] = m_max;
  }

  const float lt = l_run + xor32(l_run);
  if (my_row >= nrows) return;
  const int h = kvh * g + (my_row - my_t * g);
  const float m_out = m_run;
  if (p.splits == 1) {
    const float inv = 1.0f / lt;
    __bf16 *op = (__bf16 *)p.o + (((int64_t)b * Sq + my_t) * Hq + h) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(op + dt * 32 + jj * 8 + G * 4, oacc[dt][jj * 4 + 0] * inv, oacc[dt][jj * 4 + 1] * inv,
               oacc[dt][jj * 4 + 2] * inv, oacc[dt][jj * 4 + 3] * inv);
    if (G == 0 && p.lse != nullptr) p.lse[((int64_t)b * Hq + h) * Sq + my_t] = (m_out + log2f(lt)) * kLn2;
  } else {
    const int64_t prow = (((int64_t)split * p.B + b) * Hkv + kvh) * nrows + my_row;
    const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
    float *op = p.part_o + prow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(op + dt * 32 + jj * 8 + G * 4, oacc[dt][jj * 4 + 0] * inv, oacc[dt][jj * 4 + 1] * inv,
               oacc[dt][jj * 4 + 2] * inv, oacc[dt][jj * 4 + 3] * inv);
    if (G == 0) p.part_lse[prow] = lt > 0.0f ? (m_out + log2f(lt)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------------------
// dQ (query-stationary).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kFastThreads) void dq_bf16_kernel(DqParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int TB = kKT * D * 2;
  __shared__ __attribute__((aligned(1024))) char kb0[TB];
  __shared__ __attribute__((aligned(1024))) char vb0[TB];
  __shared__ __attribute__((aligned(1024))) char kb1[TB];
  __shared__ __attribute__((aligned(1024))) char vb1[TB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = lane >> 5, n = lane & 31;
  int bid = blockIdx.x;
  const int qblk = __builtin_amdgcn_readfirstlane(bid % p.nqblk);
  bid /= p.nqblk;
  const int kvh = __builtin_amdgcn_readfirstlane(bid % p.Hkv);
  bid /= p.Hkv;
  const int split = __builtin_amdgcn_readfirstlane(bid % p.splits);
  const int b = __builtin_amdgcn_readfirstlane(bid / p.splits);

  const int g = p.g, Sq = p.Sq, Hkv = p.Hkv, Hq = Hkv * g, nrows = p.nrows;
  const int wg_row0 = qblk * kFastRowsPerWg;
  const int wg_row1 = min(nrows, wg_row0 + kFastRowsPerWg);
  const int row0 = wg_row0 + wave * kFastRowsPerWave;
  const bool wave_active = row0 < nrows;
  const int wave_t_lo = row0 / g;
  const int wave_t_hi = (min(row0 + kFastRowsPerWave, nrows) - 1) / g;
  const int wg_t_hi = (wg_row1 - 1) / g;
  const int my_row = row0 + n;
  const int my_t = my_row / g;
  const float c = p.scale_log2;
  RowOffsets<D> ro;
  ro.init(n, G);
  TrOffsets<D> to;
  to.init(lane);

  bf16x8 qf[NSTEP], df[NSTEP];
  float lse2r = INFINITY, dvr = 0.0f;
  if (my_row < nrows) {
    const int64_t off = (((int64_t)b * Sq + my_t) * Hq + kvh * g + (my_row - my_t * g)) * D;
    const __bf16 *qp = (const __bf16 *)p.q + off;
    const __bf16 *dp = (const __bf16 *)p.d_o + off;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      qf[st] = *reinterpret_cast<const bf16x8 *>(qp + st * 16 + G * 8);
      df[st] = *reinterpret_cast<const bf16x8 *>(dp + st * 16 + G * 8);
    }
    const int64_t pk = ((int64_t)b * Hkv + kvh) * nrows + my_row;
    lse2r = p.lse2[pk];
    dvr = p.dvec[pk];
  } else {
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      qf[st] = Mma<__bf16>::zero();
      df[st] = Mma<__bf16>::zero();
    }
  }
  f32x16 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = zero16();

  const DevRow row = load_const(p.rows, b);
  const int ptiles = __builtin_amdgcn_readfirstlane(row.prefix_tiles);
  const int ntiles = ptiles + wg_t_hi / kKT + 1;
  const int tb = __builtin_amdgcn_readfirstlane((int)((int64_t)ntiles * split / p.splits));
  const int te = __builtin_amdgcn_readfirstlane((int)((int64_t)ntiles * (split + 1) / p.splits));
  TileTable tt;
  tt.init(p.tiles, row, kvh);

  auto issue = [&](const TileInfo &ti, char *kb, char *vb) __attribute__((always_inline)) {
    dma_tile<D, kKT, kNW>(kb, ti.kp, [&](int r) { return r * ti.st; }, ti.nvalid, wave, lane);
    dma_tile<D, kKT, kNW>(vb, ti.vp, [&](int r) { return r * ti.st; }, ti.nvalid, wave, lane);
  };

  auto compute = [&](const TileInfo &ti, const char *kb, const char *vb) __attribute__((always_inline)) {
    if (!wave_active) return;
    if (ti.self0 >= 0 && ti.self0 > wave_t_hi) return;
    const bool need_mask = (ti.nvalid < kKT) || (ti.self0 >= 0 && ti.self0 + kKT - 1 > wave_t_lo);
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      f32x16 sa = zero16(), dpa = zero16();
#pragma unroll
      for (int st = 0; st < NSTEP; ++st) {
        sa = Mma<__bf16>::run(row_frag_at<D>(kb, ro, 32 * sub, st), qf[st], sa);
        dpa = Mma<__bf16>::run(row_frag_at<D>(vb, ro, 32 * sub, st), df[st], dpa);
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float pv = fast_exp2(fmaf(sa[j], c, -lse2r));
        if (need_mask) {
          const int key = 32 * sub + crow(j, G);
          const bool ok = key < ti.nvalid && (ti.self0 < 0 || ti.self0 + key <= my_t);
          pv = ok ? pv : 0.0f;
        }
        sa[j] = pv * (dpa[j] - dvr);
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16x8 dsf = pack_bf16x8(sa, s);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          acc[dt] = Mma<__bf16>::run(tr_frag_at<D>(kb, to, 32 * sub + 16 * s, dt), dsf, acc[dt]);
      }
    }
  };

  if (tb < te) {
    TileInfo cur = tt.at(tb);
    issue(cur, kb0, vb0);
    __syncthreads();
    for (int it = tb; it < te; it += 2) {
      TileInfo nxt;
      const bool has1 = it + 1 < te;
      if (has1) {
        nxt = tt.at(it + 1);
        issue(nxt, kb1, vb1);
      }
      compute(cur, kb0, vb0);
      __syncthreads();
      if (!has1) break;
      const bool has2 = it + 2 < te;
      if (has2) {
        cur = tt.at(it + 2);
        issue(cur, kb0, vb0);
      }
      compute(nxt, kb1, vb1);
      __syncthreads();
    }
  }

  if (my_row >= nrows) return;
  const int h = kvh * g + (my_row - my_t * g);
  if (p.splits == 1) {
    const float sc = p.scale;
    __bf16 *op = (__bf16 *)p.dq + (((int64_t)b * Sq + my_t) * Hq + h) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(op + dt * 32 + jj * 8 + G * 4, acc[dt][jj * 4 + 0] * sc, acc[dt][jj * 4 + 1] * sc,
               acc[dt][jj * 4 + 2] * sc, acc[dt][jj * 4 + 3] * sc);
  } else {
    const int64_t prow = (((int64_t)split * p.B + b) * Hkv + kvh) * nrows + my_row;
    float *op = p.part_dq + prow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(op + dt * 32 + jj * 8 + G * 4, acc[dt][jj * 4 + 0], acc[dt][jj * 4 + 1],
               acc[dt][jj * 4 + 2], acc[dt][jj * 4 + 3]);
  }
}

// ---------------------------------------------------------------------------
// dK / dV (key-stationary). 128 keys per workgroup, resident in LDS; wave w
// owns keys 32*(w%4) .. +32 and query subtile w/4 of every 64-row block. The
// two waves sharing keys add their sums through LDS at the end.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kFastThreads) void dkdv_bf16_kernel(DkdvParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int QB = 64;
  constexpr int KTB = kDkdvKeyTile;            // 128
  constexpr int KVB = KTB * D * 2;
  constexpr int QBB = QB * D * 2;
  __shared__ __attribute__((aligned(1024))) char ktile[KVB];
  __shared__ __attribute__((aligned(1024))) char vtile[KVB];
  __shared__ __attribute__((aligned(1024))) char qb0[QBB];
  __shared__ __attribute__((aligned(1024))) char ob0[QBB];
  __shared__ __attribute__((aligned(1024))) char qb1[QBB];
  __shared__ __attribute__((aligned(1024))) char ob1[QBB];
  __shared__ __attribute__((aligned(256))) float ls0[QB];
  __shared__ __attribute__((aligned(256))) float dv0[QB];
  __shared__ __attribute__((aligned(256))) float ls1[QB];
  __shared__ __attribute__((aligned(256))) float dv1[QB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = lane >> 5, n = lane & 31;
  const int kq = wave & 3, qs = wave >> 2;     // key quarter, query subtile
  const int tile = blockIdx.x, kvh = blockIdx.y;
  const int g = p.g, Sq = p.Sq, Hkv = p.Hkv, Hq = Hkv * g, nrows = p.nrows;
  const float c = p.scale_log2;

  const __bf16 *kbase;
  const __bf16 *vbase;
  __bf16 *dkp;
  __bf16 *dvp;
  int64_t st;
  int klen, key0, use_b = 0, use_e = 1;
  const bool self = tile >= p.cart_tiles;
  int self_b = 0;
  if (!self) {
    int lo = 0, hi = p.n_carts - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (load_const(p.carts, mid).tile_begin <= tile) lo = mid; else hi = mid - 1;
    }
    const DevCart cd = load_const(p.carts, lo);
    key0 = (tile - cd.tile_begin) * KTB;
    klen = cd.len;
    kbase = (const __bf16 *)cd.k + kvh * cd.stride_head;
    vbase = (const __bf16 *)cd.v + kvh * cd.stride_head;
    dkp = cd.dk ? (__bf16 *)cd.dk + kvh * cd.stride_head : nullptr;
    dvp = cd.dv ? (__bf16 *)cd.dv + kvh * cd.stride_head : nullptr;
    st = cd.stride_tok;
    use_b = cd.use_begin;
    use_e = cd.use_end;
  } else {
    const int rel = tile - p.cart_tiles;
    self_b = rel / p.self_tiles;
    key0 = (rel % p.self_tiles) * KTB;
    klen = Sq;
    const int64_t base = ((int64_t)self_b * Sq * Hkv + kvh) * D;
    kbase = (const __bf16 *)p.k_self + base;
    vbase = (const __bf16 *)p.v_self + base;
    dkp = p.dk_self ? (__bf16 *)p.dk_self + base : nullptr;
    dvp = p.dv_self ? (__bf16 *)p.dv_self + base : nullptr;
    st = (int64_t)Hkv * D;
  }
  const int nk = min(KTB, klen - key0);           // valid keys of this tile (>= 1)
  const int wkey = kq * 32;                       // wave's first key within the tile
  const int my_key = wkey + n;                    // lane's key within the tile
  const bool key_ok = my_key < nk;
  const bool wave_has_keys = wkey < nk;
  const int abs_key = key0 + my_key;              // for the causal test on self keys
  RowOffsets<D> ro;
  ro.init(n, G);
  TrOffsets<D> to;
  to.init(lane);

  // Stage this workgroup's K and V once.
  {
    const int sti = (int)st;
    dma_tile<D, KTB, kNW>(ktile, kbase + (int64_t)key0 * st, [&](int r) { return r * sti; }, nk, wave, lane);
    dma_tile<D, KTB, kNW>(vtile, vbase + (int64_t)key0 * st, [&](int r) { return r * sti; }, nk, wave, lane);
  }

  f32x16 dk[DT], dv[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    dk[dt] = zero16();
    dv[dt] = zero16();
  }

  const int nqb = (nrows + QB - 1) / QB;
  const int qb_first = self ? (key0 * g) / QB : 0;
  const int per_use = nqb - qb_first;
  const int nblk = per_use * (use_e - use_b);

  auto block_src = [&](int blk, int &b, int &qb) __attribute__((always_inline)) {
    const int u = blk / per_use;
    qb = qb_first + (blk - u * per_use);
    b = self ? self_b : load_const(p.uses, __builtin_amdgcn_readfirstlane(use_b + u));
  };
  auto issue = [&](int blk, char *qb_l, char *ob_l, float *ls_l, float *dv_l) __attribute__((always_inline)) {
    int b, qb;
    block_src(blk, b, qb);
    const int r0 = qb * QB;
    const int nv = min(QB, nrows - r0);
    // Packed row r0 + r is query position t = (r0+r)/g, head (r0+r)%g of the
    // group; offsets are taken from the block's first position.
    const int t0 = r0 / g;
    const int64_t head0 = (((int64_t)b * Sq + t0) * Hq + kvh * g) * D;
    auto rowoff = [&](int r) __attribute__((always_inline)) {
      const int rr = r0 + r, t = rr / g;
      return ((t - t0) * Hq + (rr - t * g)) * D;
    };
    dma_tile<D, QB, kNW>(qb_l, (const __bf16 *)p.q + head0, rowoff, nv, wave, lane);
    dma_tile<D, QB, kNW>(ob_l, (const __bf16 *)p.d_o + head0, rowoff, nv, wave, lane);
    if (wave == 0) {
      // rows >= nrows read a clamped in-range row and are masked in compute
      const int64_t base = ((int64_t)b * Hkv + kvh) * nrows + r0;
      dma_f32x64(ls_l, p.lse2 + base, nv, lane);
      dma_f32x64(dv_l, p.dvec + base, nv, lane);
    }
  };
  auto compute = [&](int blk, const char *qb_l, const char *ob_l, const float *ls_l, const float *dv_l) __attribute__((always_inline)) {
    if (!wave_has_keys) return;
    int b, qb;
    block_src(blk, b, qb);
    (void)b;
    const int r0 = qb * QB;
    const int sub_r0 = r0 + 32 * qs;                 // first packed row of this wave's subtile
    if (sub_r0 >= nrows) return;
    const int t_hi = (min(sub_r0 + 32, nrows) - 1) / g;
    if (self && key0 + wkey > t_hi) return;
    const bool need_mask = (sub_r0 + 32 > nrows) || !key_ok || (self && key0 + wkey + 31 > sub_r0 / g);
    f32x16 sa = zero16(), dpa = zero16();
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      sa = Mma<__bf16>::run(row_frag_at<D>(qb_l, ro, 32 * qs, s), row_frag_at<D>(ktile, ro, wkey, s), sa);
      dpa = Mma<__bf16>::run(row_frag_at<D>(ob_l, ro, 32 * qs, s), row_frag_at<D>(vtile, ro, wkey, s), dpa);
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int ql = 32 * qs + crow(j, G);           // query row within the block
      float pv = fast_exp2(fmaf(sa[j], c, -ls_l[ql]));
      if (need_mask) {
        const int rr = r0 + ql;
        bool ok = key_ok && rr < nrows;
        if (self) ok = ok && abs_key <= rr / g;
        pv = ok ? pv : 0.0f;
      }
      sa[j] = pv;
      dpa[j] = pv * (dpa[j] - dv_l[ql]);
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const bf16x8 pf = pack_bf16x8(sa, s), dsf = pack_bf16x8(dpa, s);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        dv[dt] = Mma<__bf16>::run(tr_frag_at<D>(ob_l, to, 32 * qs + 16 * s, dt), pf, dv[dt]);
        dk[dt] = Mma<__bf16>::run(tr_frag_at<D>(qb_l, to, 32 * qs + 16 * s, dt), dsf, dk[dt]);
      }
    }
  };

  if (nblk > 0) {
    issue(0, qb0, ob0, ls0, dv0);
    __syncthreads();
    for (int blk = 0; blk < nblk; blk += 2) {
      const bool has1 = blk + 1 < nblk;
      if (has1) issue(blk + 1, qb1, ob1, ls1, dv1);
      compute(blk, qb0, ob0, ls0, dv0);
      __syncthreads();
      if (!has1) break;
      if (blk + 2 < nblk) issue(blk + 2, qb0, ob0, ls0, dv0);
      compute(blk + 1, qb1, ob1, ls1, dv1);
      __syncthreads();
    }
  } else {
    __syncthreads();
  }

  // Pairwise reduction: waves 4..7 hand their sums to waves 0..3 through the
  // K tile, which is no longer read: PD accumulators of 4 waves per pass.
  constexpr int PD = KVB / (4 * 64 * 16 * 4);
  static_assert(PD >= 1 && DT % PD == 0, "reduction pass size");
  float *red = reinterpret_cast<float *>(ktile);
#pragma unroll
  for (int pass = 0; pass < 2 * (DT / PD); ++pass) {
    f32x16 *acc = pass < DT / PD ? dk : dv;
    const int d0 = (pass % (DT / PD)) * PD;
    if (qs == 1) {
#pragma unroll
      for (int i = 0; i < PD; ++i)
        *reinterpret_cast<f32x16 *>(red + ((kq * PD + i) * 64 + lane) * 16) = acc[d0 + i];
    }
    __syncthreads();
    if (qs == 0) {
#pragma unroll
      for (int i = 0; i < PD; ++i)
        acc[d0 + i] += *reinterpret_cast<const f32x16 *>(red + ((kq * PD + i) * 64 + lane) * 16);
    }
    __syncthreads();
  }
  if (qs != 0 || !key_ok) return;
  const float sc = p.scale;
  const int64_t krow = (int64_t)(key0 + my_key) * st;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d0 = dt * 32 + jj * 8 + G * 4;
      if (dkp)
        store4(dkp + krow + d0, dk[dt][jj * 4 + 0] * sc, dk[dt][jj * 4 + 1] * sc, dk[dt][jj * 4 + 2] * sc,
               dk[dt][jj * 4 + 3] * sc);
      if (dvp)
        store4(dvp + krow + d0, dv[dt][jj * 4 + 0], dv[dt][jj * 4 + 1], dv[dt][jj * 4 + 2], dv[dt][jj * 4 + 3]);
    }
}

hipError_t launch_fwd_bf16(const FwdParams &p, int D, hipStream_t s) {
  const int64_t grid = (int64_t)p.nqblk * p.Hkv * p.splits * p.B;
  if (D == 64) {
    hipLaunchKernelGGL((fwd_bf16_kernel<64, false>), dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
    hipLaunchKernelGGL((fwd_bf16_kernel<64, true>), dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
  } else {
    hipLaunchKernelGGL((fwd_bf16_kernel<128, false>), dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
    hipLaunchKernelGGL((fwd_bf16_kernel<128, true>), dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_dq_bf16(const DqParams &p, int D, hipStream_t s) {
  const int64_t grid = (int64_t)p.nqblk * p.Hkv * p.splits * p.B;
  if (D == 64)
    hipLaunchKernelGGL(dq_bf16_kernel<64>, dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
  else
    hipLaunchKernelGGL(dq_bf16_kernel<128>, dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_dkdv_bf16(const DkdvParams &p, int D, int gx, hipStream_t s) {
  if (D == 64)
    hipLaunchKernelGGL(dkdv_bf16_kernel<64>, dim3((unsigned)gx, (unsigned)p.Hkv), dim3(kFastThreads), 0, s, p);
  else
    hipLaunchKernelGGL(dkdv_bf16_kernel<128>, dim3((unsigned)gx, (unsigned)p.Hkv), dim3(kFastThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace cas
