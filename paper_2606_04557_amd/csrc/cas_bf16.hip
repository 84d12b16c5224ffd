// bf16 fast path of multi-cartridge prefix attention for gfx950.
//
// All three kernels use 512-thread workgroups (8 waves, two per SIMD, so one
// wave's VALU work overlaps the other's MFMA work), swizzled row tiles in LDS
// filled by asynchronous direct global->LDS copies and double buffering. An
// operand reduced along its row axis comes from ds_read_b64_tr_b16 (V in the
// forward, K in dQ) or, in dK/dV, from transposed copies of Q and dO that a
// prologue kernel writes once per backward.
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
constexpr int kDkdvLead = 6;           // dK/dV: LDS fragments in flight ahead of their MFMA
constexpr int kDkdvPrio = 1;           // dK/dV: wave priority in a matrix phase (0 in VALU phases)
constexpr int kRefMargin = 64;         // forward: row sums below 2^kRefMargin need no exact pass

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
#pragma unroll
    for (int i = 0; i < PER; ++i) issue_one(tile, base, st, nvalid, wave, i);
  }
  // Instruction i (< PER) of this wave's share only.
  __device__ __forceinline__ void issue_one(char *tile, const __bf16 *base, int st, int nvalid, int wave,
                                            int i) const {
    issue_rs(tile, make_rsrc(base, ((nvalid - 1) * st + D) * 2), st, nvalid, wave, i);
  }
  // The same through a given resource (an empty one writes zeros).
  __device__ __forceinline__ void issue_rs(char *tile, BufRsrc rs, int st, int nvalid, int wave, int i) const {
    const int inst = wave + i * NW;
    if (NI % NW == 0 || inst < NI) dma16(rs, (min(row[i], nvalid - 1) * st + coff[i]) * 2, tile + inst * 1024);
  }
};

// Pins register values at this point: the compiler may not move their
// computation past it (e.g. across a barrier into the next phase).
template <typename T, int N>
__device__ __forceinline__ void fence_regs(T (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}

// Workgroup barrier that orders LDS use: this wave's LDS reads have returned,
// and the compiler moves no memory access across it. Outstanding direct
// global->LDS copies are not waited for (wait_vmcnt does that).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt, expcnt untouched
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// The dK/dV order entry of this workgroup when the lists are per XCD
// (DevQueue): workgroup j of XCD x takes entry j of the XCD's static head;
// past the head, thread 0 claims the next tail entry with an atomic counter,
// of its own XCD first, then of the XCD with the most unclaimed entries
// left, and the workgroup reads it from LDS. -1: nothing left. Every tail
// entry is claimed exactly once: each XCD launches at least as many tail
// workgroups as its tail holds, and each tries its own tail first.
__device__ __forceinline__ int dkdv_entry(const DkdvParams &p, int tid, int &slot) {
  const int X = p.xcds;
  const int x = (int)blockIdx.x % X, j = (int)blockIdx.x / X;
  const DevQueue own = load_const(p.queues, x);
  if (j < own.head) return own.off + j;
  if (tid == 0) {
    int e = -1, y = x;
    for (int attempt = 0; attempt < 2 * X && e < 0; ++attempt) {
      if (attempt > 0) {
        int best = -1, most = 0;
        for (int z = 0; z < X; ++z) {
          const DevQueue qz = p.queues[z];
          const int left = (qz.cnt - qz.head) - __hip_atomic_load(p.claim + z, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (left > most) {
            most = left;
            best = z;
          }
        }
        if (best < 0) break;
        y = best;
      }
      const DevQueue qy = p.queues[y];
      const int i = __hip_atomic_fetch_add(p.claim + y, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (i < qy.cnt - qy.head) e = qy.off + qy.head + i;
    }
    slot = e;
  }
  __syncthreads();
  return __builtin_amdgcn_readfirstlane(slot);
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
// which it sees a key (the only tile whose row maximum is computed), and never
// moved, so O is never rescaled in the loop and later tiles need no maximum.
// Later scores may exceed m: while the row sum stays below 2^kRefMargin every
// P, every partial sum and O stay far inside fp32 and bf16 range. A row whose
// sum reaches it (or overflows) flags its workgroup, and a second launch
// (FIXUP) recomputes only the flagged workgroups with the exact online
// softmax (running maximum, O and the sum rescaled at every tile). Unflagged
// workgroups of the second launch exit at once.
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
  // The host lists the workgroups in dispatch order: per XCD, whole KV heads
  // where they divide evenly, longest first.
  const DevItem item = load_const(p.items, (int)blockIdx.x);
  const int qblk = __builtin_amdgcn_readfirstlane(item.qblk);
  const int split = __builtin_amdgcn_readfirstlane(item.split);
  const int b = __builtin_amdgcn_readfirstlane(item.b);
  const int kvh = __builtin_amdgcn_readfirstlane(item.kvh);
  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g;
  const DevRow row = load_const(p.rows, b);
  const int tok0 = __builtin_amdgcn_readfirstlane(row.tok0);
  const int nrows = __builtin_amdgcn_readfirstlane(row.len) * g;
  const int wg_row0 = qblk * kFastRowsPerWg;
  if (wg_row0 >= nrows) return;   // (the host lists only blocks with rows)
  if constexpr (FIXUP) {
    if (load_const(p.ovf_flag, (int)blockIdx.x) == 0) return;
  }

  const int wg_row1 = min(nrows, wg_row0 + kFastRowsPerWg);
  const int row0 = wg_row0 + wave * kFastRowsPerWave;
  const bool wave_active = row0 < nrows;
  const int wave_t_lo = row0 / g;
  const int wave_t_hi = (min(row0 + kFastRowsPerWave, nrows) - 1) / g;
  const int wg_t_hi = (wg_row1 - 1) / g;
  const int my_row = row0 + n;
  const int my_t = my_row / g;
  const float c = p.scale_log2;

  // Wave-uniform tile range of this split (readfirstlane keeps it, and every
  // tile-table read that depends on it, in scalar registers).
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
    const __bf16 *rp = (const __bf16 *)p.q + (((int64_t)tok0 + my_t) * Hq + kvh * g + (my_row - my_t * g)) * D;
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
  // (FIXUP) the running row maximum.
  float m_run = -INFINITY;
  float l_run = 0.0f;

  // Group B's share of every tile copy (4 waves).
  CopyLanes<D, kKT, 4> cl;
  cl.init(wave & 3, lane);
  constexpr int kCopyInst = CopyLanes<D, kKT, 4>::PER;   // per wave per K or V tile
  constexpr int kPieces = 2 * kCopyInst;                   // copy instructions per softmax phase
  static_assert(16 % kPieces == 0, "copy pieces spread over the 16 exponential pairs");

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
  float alpha = 1.0f;   // FIXUP: O rescale factor of the current tile
  // piece(n), n < kPieces: copy instruction n of the phase (group B's tile
  // copies), spread evenly over the exponentials.
  auto softmax = [&](auto MASK, int lim, auto &&piece) __attribute__((always_inline)) {
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
    auto tile_max = [&]() __attribute__((always_inline)) {
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 16; j += 2) mx = fmaxf(fmaxf(mx, fmaxf(s0[j], s1[j])), fmaxf(s0[j + 1], s1[j + 1]));
      return fmaxf(mx, xor32(mx)) * c;
    };
    if constexpr (!FIXUP) {
      // Only until every row of the wave has seen a key.
      if (wave_any(m_run == -INFINITY)) {
        const float mt = tile_max();
        m_run = (m_run == -INFINITY) ? mt : m_run;
      }
    } else {
      // Running maximum; the sum is rescaled here, O by the caller (outside
      // its branches, so the accumulators are written in one place).
      const float m_new = fmaxf(m_run, tile_max());
      alpha = (m_new == -INFINITY) ? 1.0f : fast_exp2(m_run - m_new);
      l_run *= alpha;
      m_run = m_new;
    }
    const float mu = (m_run == -INFINITY) ? 0.0f : m_run;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      s0[j] = fast_exp2(fmaf(s0[j], c, -mu));
      s1[j] = fast_exp2(fmaf(s1[j], c, -mu));
      constexpr int EPP = 16 / kPieces;
      if (j % EPP == EPP - 1) {
        asm volatile("" : "+v"(s0[j]), "+v"(s1[j]));   // keep the copies spread
        piece(j / EPP);
      }
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
  auto xphase_body = [&](int j, auto &&piece) __attribute__((always_inline)) {
    auto all_pieces = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int n = 0; n < kPieces; ++n) piece(n);
    };
    if (j < 0 || j >= nt) {
      all_pieces();
      return;
    }
    if (!live(j)) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int s = 0; s < 2; ++s) pf[a][s] = Mma<__bf16>::zero();
      all_pieces();
      return;
    }
    const int self0 = self0_of(j);
    const int nvalid = __builtin_amdgcn_readfirstlane(tt.nvalid(tb + j));
    if (nvalid < kKT || (self0 >= 0 && self0 + kKT - 1 > wave_t_lo)) {
      const int lim = self0 < 0 ? nvalid - 1 : min(nvalid - 1, my_t - self0);
      softmax(std::true_type{}, lim, piece);
    } else {
      softmax(std::false_type{}, kKT - 1, piece);
    }
  };
  auto xphase = [&](int j, auto &&piece) __attribute__((always_inline)) {
    if constexpr (FIXUP) alpha = 1.0f;
    xphase_body(j, piece);
    if constexpr (FIXUP) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
    }
  };

  // Group B's copies. tk: the K tile issued last (tile i+1 when phase 2i
  // starts), whose V is issued next.
  TileInfo tk;
  auto copy_k = [&](char *kbn, int j) __attribute__((always_inline)) {
    tk = tt.at(tb + j);
    cl.issue(kbn, tk.kp, tk.st, tk.nvalid, wave & 3);
  };
  auto no_piece = [](int) {};
  // Phase 2i: V_{i+1} and K_{i+2}, spread over the softmax of tile i-1 (copies
  // past the last tile go through an empty resource and write zeros into
  // buffers nothing reads); at its end the copies of phase 2i-2 are waited for.
  auto even_b = [&](int i, char *kbn, char *vbn) __attribute__((always_inline)) {
    const TileInfo tv = tk;                                   // tile i+1 (or the last)
    const TileInfo tn = tt.at(tb + min(i + 2, nt - 1));
    const BufRsrc rv = make_rsrc(tv.vp, i + 1 < nt ? ((tv.nvalid - 1) * tv.st + D) * 2 : 0);
    const BufRsrc rk = make_rsrc(tn.kp, i + 2 < nt ? ((tn.nvalid - 1) * tn.st + D) * 2 : 0);
    xphase(i - 1, [&](int n) __attribute__((always_inline)) {
      if (n < kCopyInst) cl.issue_rs(vbn, rv, tv.st, tv.nvalid, wave & 3, n);
      else cl.issue_rs(kbn, rk, tn.st, tn.nvalid, wave & 3, n - kCopyInst);
    });
    tk = tn;
    wait_vmcnt<2 * kCopyInst>();
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
        if constexpr (A) gphase(i, kbi, vbp);
        else even_b(i, kbn, vbn);
        lds_barrier();
      };
      auto odd = [&](int i, const char *kbi, const char *vbp) __attribute__((always_inline)) {
        if constexpr (A) xphase(i, no_piece);
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
    wait_vmcnt<0>();
  }
  if constexpr (!FIXUP) {
    // Every wave reaches this point: flag the workgroup if a row sum reached
    // 2^kRefMargin or overflowed (exponent field also catches inf and NaN).
    const unsigned eb = (__float_as_uint(l_run) >> 23) & 0xffu;
    const int any = __syncthreads_or(eb >= 127u + (unsigned)kRefMargin ? 1 : 0);
    if (tid == 0) p.ovf_flag[blockIdx.x] = any;
  }

  const float lt = l_run + xor32(l_run);
  if (my_row >= nrows) return;
  const int h = kvh * g + (my_row - my_t * g);
  const float m_out = m_run;
  if (p.splits == 1) {
    const float inv = 1.0f / lt;
    __bf16 *op = (__bf16 *)p.o + (((int64_t)tok0 + my_t) * Hq + h) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(op + dt * 32 + jj * 8 + G * 4, oacc[dt][jj * 4 + 0] * inv, oacc[dt][jj * 4 + 1] * inv,
               oacc[dt][jj * 4 + 2] * inv, oacc[dt][jj * 4 + 3] * inv);
    if (G == 0 && p.lse != nullptr)
      p.lse[(int64_t)row.lse0 + (int64_t)h * p.lse_hs + my_t] = (m_out + log2f(lt)) * kLn2;
  } else {
    const int64_t prow = split * p.plane + (int64_t)tok0 * Hq + kvh * nrows + my_row;
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
// dQ (query-stationary): ping-pong between the two waves of each SIMD.
//
// The key axis is walked in 32-key units (half tiles of the tile table). Per
// unit u a wave runs a matrix phase G_u (dQ^T += K_{u-1}^T dS_{u-1}^T, then
// S_u^T = K_u Q^T and dP_u^T = V_u dO^T: 24 MFMAs for d = 128 in one
// scheduling region) and a VALU phase X_u (P = exp2(S c - LSE2), masks,
// dS = P (dP - D), bf16 packing of dS). Waves 0-3 (group A) run G_u while
// waves 4-7 (group B) run X_{u-1}, and the other way round in the next phase;
// every phase ends in a workgroup barrier, so on each SIMD one wave's MFMA
// stream runs beside the other wave's VALU work. (32-key units keep the
// scores, dP and dS of one unit within the 256 registers of a wave that
// shares its SIMD.)
//
// LDS: four K and four V unit buffers, unit u in buffer u % 4. K_u is read by
// G_u and G_{u+1} (up to phase 2u+3), V_u by G_u (up to phase 2u+1). Only
// group B copies: at the start of phase 2u (a VALU phase for it) it issues
// unit u+2 into the buffers unit u-2 left free, and at the end of phase 2u it
// waits for unit u+1, which G_{u+1} reads from phase 2u+2 on.
// ---------------------------------------------------------------------------
constexpr int kDqUnit = 32;   // keys per dQ unit

template <int D>
__global__ __launch_bounds__(kFastThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dq_bf16_kernel(DqParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int UB = kDqUnit * D * 2;   // bytes per unit buffer
  __shared__ __attribute__((aligned(1024))) char kb0[UB];
  __shared__ __attribute__((aligned(1024))) char kb1[UB];
  __shared__ __attribute__((aligned(1024))) char kb2[UB];
  __shared__ __attribute__((aligned(1024))) char kb3[UB];
  __shared__ __attribute__((aligned(1024))) char vb0[UB];
  __shared__ __attribute__((aligned(1024))) char vb1[UB];
  __shared__ __attribute__((aligned(1024))) char vb2[UB];
  __shared__ __attribute__((aligned(1024))) char vb3[UB];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int G = lane >> 5, n = lane & 31;
  // The host lists the workgroups in dispatch order: per XCD, whole KV heads
  // where they divide evenly, longest first.
  const DevItem item = load_const(p.items, (int)blockIdx.x);
  const int qblk = __builtin_amdgcn_readfirstlane(item.qblk);
  const int split = __builtin_amdgcn_readfirstlane(item.split);
  const int b = __builtin_amdgcn_readfirstlane(item.b);
  const int kvh = __builtin_amdgcn_readfirstlane(item.kvh);

  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g;
  const DevRow row = load_const(p.rows, b);
  const int tok0 = __builtin_amdgcn_readfirstlane(row.tok0);
  const int nrows = __builtin_amdgcn_readfirstlane(row.len) * g;
  const int wg_row0 = qblk * kFastRowsPerWg;
  if (wg_row0 >= nrows) return;   // (the host lists only blocks with rows)
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
  float lse2r = INFINITY, ndr = 0.0f;
  if (my_row < nrows) {
    const int64_t off = (((int64_t)tok0 + my_t) * Hq + kvh * g + (my_row - my_t * g)) * D;
    const __bf16 *qp = (const __bf16 *)p.q + off;
    const __bf16 *dp = (const __bf16 *)p.d_o + off;
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      qf[st] = *reinterpret_cast<const bf16x8 *>(qp + st * 16 + G * 8);
      df[st] = *reinterpret_cast<const bf16x8 *>(dp + st * 16 + G * 8);
    }
    const int64_t pk = (int64_t)tok0 * Hq + kvh * nrows + my_row;
    lse2r = p.lse2[pk];
    ndr = p.nd[pk];
  } else {
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
      qf[st] = Mma<__bf16>::zero();
      df[st] = Mma<__bf16>::zero();
    }
  }
  // Unit copies are waited for with partial vmcnt counts, which must not
  // include these loads.
  wait_vmcnt<0>();

  f32x16 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = zero16();

  const int ptiles = __builtin_amdgcn_readfirstlane(row.prefix_tiles);
  const int ntiles = ptiles + wg_t_hi / kKT + 1;
  const int tb = __builtin_amdgcn_readfirstlane((int)((int64_t)ntiles * split / p.splits));
  const int te = __builtin_amdgcn_readfirstlane((int)((int64_t)ntiles * (split + 1) / p.splits));
  const int nu = 2 * (te - tb);   // units of this split
  TileTable tt;
  tt.init(p.tiles, row, kvh);

  // Unit u: half u % 2 of local tile u / 2.
  struct Unit {
    const __bf16 *kp, *vp;
    int st, nvalid, self0;   // nvalid <= 0: no keys
  };
  auto unit_at = [&](int u) __attribute__((always_inline)) {
    const TileInfo t = tt.at(tb + (u >> 1));
    const int hk = (u & 1) * kDqUnit;
    Unit x;
    x.kp = t.kp + (int64_t)hk * t.st;
    x.vp = t.vp + (int64_t)hk * t.st;
    x.st = t.st;
    x.nvalid = min(kDqUnit, t.nvalid - hk);
    x.self0 = t.self0 < 0 ? -1 : t.self0 + hk;
    return x;
  };

  // Group B's share of every unit copy (4 waves): instruction k of a K or V
  // unit moves rows cr0 + RSTEP k (16 bytes per lane, swizzled chunk ccol);
  // the swizzle repeats every 16 rows, so one row and one chunk offset per
  // lane serve every instruction. Rows past nvalid re-read row nvalid-1
  // (masked later); a unit without keys goes through an empty resource.
  constexpr int CPR = D / 8;                                 // 16-byte chunks per row
  constexpr int kCopyInst = kDqUnit * CPR / 64 / 4;          // per wave per K or V unit
  constexpr int RSTEP = 4 * 64 / CPR;                        // rows between a wave's instructions
  constexpr int kPieces = 2 * kCopyInst;                     // copy instructions per VALU phase
  static_assert(kCopyInst >= 1 && kDqUnit * CPR == kCopyInst * 4 * 64, "unit copies split evenly");
  static_assert(RSTEP % 16 == 0, "swizzle period divides the row step");
  static_assert(16 % kPieces == 0, "copy pieces spread over the 16 exponentials");
  const int cpos = (wave & 3) * 64 + lane;
  const int cr0 = cpos / CPR;
  const int ccol = ((cpos % CPR) ^ swz<D>(cr0)) * 8;
  auto copy_one = [&](char *buf, const BufRsrc &rs, const Unit &x, int k) __attribute__((always_inline)) {
    dma16(rs, (min(cr0 + RSTEP * k, max(x.nvalid, 1) - 1) * x.st + ccol) * 2, buf + ((wave & 3) + 4 * k) * 1024);
  };
  auto unit_bytes = [&](const Unit &x, bool has) __attribute__((always_inline)) {
    return (has && x.nvalid > 0) ? ((x.nvalid - 1) * x.st + D) * 2 : 0;
  };

  // S^T and dP^T of the unit between its G and X phases; dS^T of the unit
  // (bf16, per 16-key step) between its X phase and the next G phase.
  f32x16 sa = zero16(), dpa = zero16();
  bf16x8 dsf[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) dsf[s] = Mma<__bf16>::zero();

  // Matrix phase as one software-pipelined MFMA sequence: dQ^T of the previous
  // unit (2*DT MFMAs, K^T fragments by two transposed LDS reads each), then
  // S^T and dP^T of this unit (2*NSTEP MFMAs, one row read each). The fragment
  // of MFMA k+LEAD is read while MFMA k runs, into a ring of LEAD+1 registers.
  auto matrix = [&](const char *kbp, const char *kb, const char *vb) __attribute__((always_inline)) {
    constexpr int NQ = 2 * DT;
    constexpr int N = NQ + 2 * NSTEP;
    constexpr int LEAD = 4, R = LEAD + 1;
    // MFMA k < NQ: 16-key step s = k / DT, dt = k % DT.
    // MFMA k >= NQ: st = (k - NQ) / 2; S (even) or dP (odd).
    auto load = [&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < NQ) {
        return tr_frag_at<D>(kbp, to, 16 * (k / DT), k % DT);
      } else {
        constexpr int st = (k - NQ) / 2;
        if constexpr ((k - NQ) % 2 == 0) return row_frag_at<D>(kb, ro, 0, st);
        else return row_frag_at<D>(vb, ro, 0, st);
      }
    };
    auto mma = [&](auto K, const bf16x8 &f) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < NQ) {
        acc[k % DT] = Mma<__bf16>::run(f, dsf[k / DT], acc[k % DT]);
      } else {
        // The first step starts from an inline zero accumulator.
        constexpr int st = (k - NQ) / 2;
        if constexpr ((k - NQ) % 2 == 0) sa = Mma<__bf16>::run(f, qf[st], st == 0 ? zero16() : sa);
        else dpa = Mma<__bf16>::run(f, df[st], st == 0 ? zero16() : dpa);
      }
    };
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
    static_for<LEAD>([&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      if constexpr (k < N) sched_ds_read<(k < NQ ? 2 : 1)>();
    });
    static_for<N>([&](auto K) __attribute__((always_inline)) {
      constexpr int k = decltype(K)::value;
      sched_mfma<1>();
      if constexpr (k + LEAD < N) sched_ds_read<(k + LEAD < NQ ? 2 : 1)>();
    });
  };

  // VALU phase of a live unit; piece(n), n < kPieces: copy instruction n of
  // the phase, spread evenly over the exponentials.
  auto dsoft = [&](auto MASK, int lim, auto &&piece) __attribute__((always_inline)) {
    if constexpr (decltype(MASK)::value) {
      // lim: last visible key of this lane's query within the unit (negative:
      // none). Register j of lane group G holds key crow(j, 0) + 4G.
      const int limg = lim - 4 * G;
#pragma unroll
      for (int j = 0; j < 16; ++j) sa[j] = crow(j, 0) <= limg ? sa[j] : -INFINITY;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      // dP accumulated from zero: dS = P (dP - D) with -D added here.
      sa[j] = fast_exp2(fmaf(sa[j], c, -lse2r)) * (dpa[j] + ndr);
      constexpr int EPP = 16 / kPieces;
      if (j % EPP == EPP - 1) {
        asm volatile("" : "+v"(sa[j]));   // keep the copies spread
        piece(j / EPP);
      }
      if (j % 8 == 7) dsf[j / 8] = pack_bf16x8(sa, j / 8);
    }
  };

  auto gphase = [&](int u, const char *kbp, const char *kb, const char *vb) __attribute__((always_inline)) {
    if (u <= nu && wave_active) matrix(kbp, kb, vb);
  };
  auto xphase = [&](int u, auto &&piece) __attribute__((always_inline)) {
    auto all_pieces = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int k = 0; k < kPieces; ++k) piece(k);
    };
    if (u < 0 || u >= nu) {
      all_pieces();
      return;
    }
    const Unit x = unit_at(u);
    if (!wave_active || x.nvalid <= 0 || (x.self0 >= 0 && x.self0 > wave_t_hi)) {
#pragma unroll
      for (int s = 0; s < 2; ++s) dsf[s] = Mma<__bf16>::zero();
      all_pieces();
      return;
    }
    if (x.nvalid < kDqUnit || (x.self0 >= 0 && x.self0 + kDqUnit - 1 > wave_t_lo)) {
      const int lim = x.self0 < 0 ? x.nvalid - 1 : min(x.nvalid - 1, my_t - x.self0);
      dsoft(std::true_type{}, lim, piece);
    } else {
      dsoft(std::false_type{}, kDqUnit - 1, piece);
    }
  };
  auto no_piece = [](int) {};

  auto issue_unit = [&](int u, char *kbn, char *vbn) __attribute__((always_inline)) {
    const Unit x = unit_at(u);
    const int bytes = unit_bytes(x, true);
    const BufRsrc rk = make_rsrc(x.kp, bytes), rv = make_rsrc(x.vp, bytes);
#pragma unroll
    for (int k = 0; k < kCopyInst; ++k) copy_one(kbn, rk, x, k);
#pragma unroll
    for (int k = 0; k < kCopyInst; ++k) copy_one(vbn, rv, x, k);
  };
  // Phase 2u for group B: unit u+2 (through empty resources past the last
  // unit: zeros into buffers that only G_nu's unused products read) spread
  // over X_{u-1}; then wait for unit u+1.
  auto even_b = [&](int u, char *kbn, char *vbn) __attribute__((always_inline)) {
    const Unit x = unit_at(min(u + 2, nu - 1));
    const int bytes = unit_bytes(x, u + 2 < nu);
    const BufRsrc rk = make_rsrc(x.kp, bytes), rv = make_rsrc(x.vp, bytes);
    xphase(u - 1, [&](int k) __attribute__((always_inline)) {
      if (k < kCopyInst) copy_one(kbn, rk, x, k);
      else copy_one(vbn, rv, x, k - kCopyInst);
    });
    wait_vmcnt<kPieces>();
  };

  if (nu > 0) {
    // G_0 multiplies K buffer 3 by dS = 0: clear it so no stale bit pattern
    // (a NaN) can reach dQ.
    for (int i = tid; i < UB / 16; i += kFastThreads) reinterpret_cast<uint4 *>(kb3)[i] = uint4{0, 0, 0, 0};
    // Prologue (group B): unit 0, then unit 1 (nu is even, so it exists).
    if (grp == 1) {
      issue_unit(0, kb0, vb0);
      wait_vmcnt<0>();
      issue_unit(1, kb1, vb1);
    }
    lds_barrier();
    // Eight phases per iteration (four units), so every buffer is a fixed LDS
    // address: G_u reads K_{u-1}, K_u and V_u from buffers (u-1)%4 and u%4;
    // the copies of phase 2u go to buffers (u+2)%4. Each group runs its own
    // copy of the loop (straight-line phases); s_barrier pairs them.
    auto run = [&](auto GROUP_A) __attribute__((always_inline)) {
      constexpr bool A = decltype(GROUP_A)::value;
      auto even = [&](int u, const char *kbp, const char *kbi, const char *vbi, char *kbn, char *vbn)
                      __attribute__((always_inline)) {
        if constexpr (A) gphase(u, kbp, kbi, vbi);
        else even_b(u, kbn, vbn);
        lds_barrier();
      };
      auto odd = [&](int u, const char *kbp, const char *kbi, const char *vbi) __attribute__((always_inline)) {
        if constexpr (A) xphase(u, no_piece);
        else gphase(u, kbp, kbi, vbi);
        lds_barrier();
      };
      for (int u = 0; u <= nu; u += 4) {
        even(u, kb3, kb0, vb0, kb2, vb2);
        odd(u, kb3, kb0, vb0);
        if (u + 1 > nu) break;
        even(u + 1, kb0, kb1, vb1, kb3, vb3);
        odd(u + 1, kb0, kb1, vb1);
        if (u + 2 > nu) break;
        even(u + 2, kb1, kb2, vb2, kb0, vb0);
        odd(u + 2, kb1, kb2, vb2);
        if (u + 3 > nu) break;
        even(u + 3, kb2, kb3, vb3, kb1, vb1);
        odd(u + 3, kb2, kb3, vb3);
      }
    };
    if (grp == 0) run(std::true_type{});
    else run(std::false_type{});
    wait_vmcnt<0>();
  }

  if (my_row >= nrows) return;
  const int h = kvh * g + (my_row - my_t * g);
  if (p.splits == 1) {
    const float sc = p.scale;
    __bf16 *op = (__bf16 *)p.dq + (((int64_t)tok0 + my_t) * Hq + h) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(op + dt * 32 + jj * 8 + G * 4, acc[dt][jj * 4 + 0] * sc, acc[dt][jj * 4 + 1] * sc,
               acc[dt][jj * 4 + 2] * sc, acc[dt][jj * 4 + 3] * sc);
  } else {
    const int64_t prow = split * p.plane + (int64_t)tok0 * Hq + kvh * nrows + my_row;
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
// bf16 backward prologue, per 64-row query block of each (batch row, KV
// head):
//  * the row statistics: -D = -rowsum(dO * O) and LSE * log2(e);
//  * Q and dO transposed to [channel][64 rows] for the dK/dV kernel, zero
//    beyond the row's last packed row. Within each 16-row group the rows are
//    stored in the order 0-3, 8-11, 4-7, 12-15, so the 8 rows that one lane
//    group of a 32x32 MFMA fragment needs (4G..4G+3 and 8+4G..8+4G+3) are
//    one 16-byte chunk.
// dO is read once for both.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_prologue_bf16_kernel(PreParams p) {
  __shared__ __attribute__((aligned(16))) __bf16 tile[64][D + 8];
  const int tid = threadIdx.x;
  const int qb = blockIdx.x % p.nqb_max;
  const int kvh = blockIdx.x / p.nqb_max, b = blockIdx.y;
  const int g = p.g, Hq = p.Hkv * g;
  const DevRow row = p.rows[b];
  const int nrows = row.len * g, nqb = (nrows + 63) / 64;
  if (qb >= nqb) return;   // grid sized for the longest row
  const int64_t blk = (int64_t)row.tblk0 + kvh * nqb + qb;
  for (int which = 0; which < 2; ++which) {
    const __bf16 *src = (const __bf16 *)(which ? p.d_o : p.q);
    __bf16 *dst = (__bf16 *)(which ? p.doT : p.qT) + blk * D * 64;
    for (int i = tid; i < 64 * D / 8; i += 256) {
      const int r = i / (D / 8), c8 = i % (D / 8);
      const int rr = qb * 64 + r;
      uint4 v = uint4{0, 0, 0, 0};
      if (rr < nrows) {
        const int t = rr / g, h = kvh * g + (rr - t * g);
        v = *reinterpret_cast<const uint4 *>(src + (((int64_t)row.tok0 + t) * Hq + h) * D + c8 * 8);
      }
      *reinterpret_cast<uint4 *>(&tile[r][c8 * 8]) = v;
    }
    __syncthreads();
    if (which == 1) {
      // -D and LSE2 of the block's rows: four lanes per row, D/4 channels each.
      constexpr int CQ = D / 4;
      const int r = tid >> 2, k = tid & 3;
      const int rr = qb * 64 + r;
      float acc = 0.0f;
      int t = 0, h = 0;
      if (rr < nrows) {
        t = rr / g;
        h = kvh * g + (rr - t * g);
        const __bf16 *op = (const __bf16 *)p.o + (((int64_t)row.tok0 + t) * Hq + h) * D + k * CQ;
#pragma unroll
        for (int c8 = 0; c8 < CQ / 8; ++c8) {
          const bf16x8 ov = *reinterpret_cast<const bf16x8 *>(op + c8 * 8);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc += (float)ov[e] * (float)tile[r][k * CQ + c8 * 8 + e];
        }
      }
      acc += __shfl_xor(acc, 1, 4);
      acc += __shfl_xor(acc, 2, 4);
      if (rr < nrows && k == 0) {
        const int64_t R = (int64_t)row.tok0 * Hq + (int64_t)kvh * nrows + rr;
        p.nd[R] = -acc;
        p.lse2[R] = p.lse[(int64_t)row.lse0 + (int64_t)h * p.lse_hs + t] * kLog2e;
      }
    }
    for (int i = tid; i < D * 8; i += 256) {
      const int d = i / 8, pg = i % 8;
      bf16x8 out;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int pos = pg * 8 + e, w = pos & 15, quad = w >> 2;
        const int sq = quad == 1 ? 2 : (quad == 2 ? 1 : quad);
        out[e] = tile[(pos & ~15) + sq * 4 + (w & 3)][d];
      }
      *reinterpret_cast<bf16x8 *>(dst + d * 64 + pg * 8) = out;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// dK / dV (key-stationary): S and dP on the two waves of each SIMD.
//
// 128 keys per workgroup of eight waves. Waves w and w+4 share SIMD w and
// keys 32w .. 32w+31. Wave w (the P wave) holds their K fragments and computes
// S = Q K^T, P = exp2(S c - LSE2) and dV^T += dO^T P; wave w+4 (the dS wave)
// holds their V fragments and computes dP = dO V^T, dS = P (dP - D) and
// dK^T += Q^T dS, taking P from the P wave through LDS. Each wave so keeps one
// 32 x D accumulator and one operand set in registers (two waves per SIMD
// fit), and per 64-row query block runs 32 MFMAs (D = 128) and one VALU pass.
// Block i is two phases, each ending in a workgroup barrier:
//   A_i: P waves:  S_{i+1}, dV += dO_i^T P_i       (MFMA)
//        dS waves: dS_i = P_i (dP_i - D_i)          (VALU)
//   B_i: dS waves: dK += Q_i^T dS_i, dP_{i+1}       (MFMA)
//        P waves:  P_{i+1} = exp2(S_{i+1} c - LSE2)  (VALU)
// so on every SIMD one wave's MFMA stream runs beside the other's VALU work.
// Every operand read is a 16-byte row read: Q and dO rows for S and dP, and
// the transposed blocks Q^T and dO^T (written by the backward prologue) for
// the dK and dV products.
//
// Copies (LDS double buffers): per block, P waves fetch dO rows of block i+2,
// Q^T_{i+1} and LSE2 of i+2; dS waves fetch Q rows of block i+2, dO^T_{i+1}
// and -D of i+2 (the statistic is stored negated and loaded straight into the
// dP accumulators, so the MFMAs deliver dP - D). A wave's row-block copies go
// into its matrix phase, one per eight MFMAs, the rest into its VALU phase.
// Copy addresses (with their segment-table loads) are prepared one VALU phase
// ahead. Copies for blocks past the end use an empty buffer resource (they
// write zeros that nothing reads).
//
// P needs no mask for keys beyond the tile (their dK / dV columns are never
// stored) or for packed rows beyond the batch row's last (Q, dO, Q^T, dO^T,
// LSE2 and D all read as zero there: P = 1 and dS = 0 add nothing). On self
// keys P = 0 for rows before the key's position.
// ---------------------------------------------------------------------------
template <int D, bool GFAST>
__global__ __launch_bounds__(kFastThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dkdv_bf16_kernel(DkdvParams p) {
  constexpr int NSTEP = D / 16;
  constexpr int DT = D / 32;
  constexpr int QB = kDkdvQBlock;              // 64 query rows per block
  constexpr int KTB = kDkdvKeyTile;            // 128 keys
  constexpr int RB = QB * D * 2;               // bytes of one 64 x D block
  constexpr int NMF = 4 * NSTEP;               // MFMAs of a wave's matrix phase
  constexpr int LEAD = kDkdvLead, RING = LEAD + 1;
  constexpr int PRIO = kDkdvPrio;
  // One LDS arena. The P waves' matrix operands (Q rows, dO^T) fill the first
  // 4 RB bytes and the dS waves' (dO rows, Q^T) the next 4 RB, so each wave
  // reaches all of its fragments from one set of lane offsets plus 16-bit
  // immediates.
  constexpr int XCH = 8 * RB;                  // P of each SIMD's 32 keys x 64 rows, 4 KiB per SIMD
  constexpr int STATS = XCH + 16384;           // LSE2 x2, D x2
  constexpr int CLAIM = STATS + 4 * QB * 4;   // claimed order entry (DevQueue lists)
  // One arena for every LDS use: a second LDS object would keep the
  // compiler from telling the direct-to-LDS copies' targets from the LDS
  // reads, and it would then wait for every outstanding copy before each read.
  __shared__ __attribute__((aligned(1024))) char smem[CLAIM + 16];
  char *const qr0 = smem, *const qr1 = smem + RB, *const ot0 = smem + 2 * RB, *const ot1 = smem + 3 * RB;
  char *const or0 = smem + 4 * RB, *const or1 = smem + 5 * RB, *const qt0 = smem + 6 * RB,
              *const qt1 = smem + 7 * RB;
  char *const xch = smem + XCH;
  float *const ls0 = reinterpret_cast<float *>(smem + STATS);
  float *const ls1 = ls0 + QB;
  float *const dv0 = ls0 + 2 * QB;
  float *const dv1 = ls0 + 3 * QB;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = lane >> 5, n = lane & 31;
  const int q = wave & 3;                      // SIMD, key quarter, index within the wave's group
  const bool pwave = wave < 4;
  int entry = (int)blockIdx.x;
  if (p.queues) {
    entry = dkdv_entry(p, tid, *reinterpret_cast<int *>(smem + CLAIM));
    if (entry < 0) return;   // every list is done
  }
  const DevWg wg = load_const(p.order, entry);
  const int tile = __builtin_amdgcn_readfirstlane(wg.tile), kvh = __builtin_amdgcn_readfirstlane(wg.kvh);
  const int g = p.g, Hkv = p.Hkv, Hq = Hkv * g;
  const float c = p.scale_log2;

  const __bf16 *kbase;
  const __bf16 *vbase;
  __bf16 *dkp;
  __bf16 *dvp;
  int64_t st;
  int klen, key0, use_b = 0, nblk_all;
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
    nblk_all = cd.nblk;
  } else {
    const int rel = tile - p.cart_tiles;
    self_b = rel / p.self_tiles;
    key0 = (rel % p.self_tiles) * KTB;
    const DevRow sr = load_const(p.rows, self_b);
    klen = sr.len;
    if (key0 >= klen) return;   // grid sized for the longest row
    const int64_t base = ((int64_t)sr.tok0 * Hkv + kvh) * D;
    kbase = (const __bf16 *)p.k_self + base;
    vbase = (const __bf16 *)p.v_self + base;
    dkp = p.dk_self ? (__bf16 *)p.dk_self + base : nullptr;
    dvp = p.dv_self ? (__bf16 *)p.dv_self + base : nullptr;
    st = (int64_t)Hkv * D;
    nblk_all = (klen * g + QB - 1) / QB - (key0 * g) / QB;
  }
  const int nk = __builtin_amdgcn_readfirstlane(min(KTB, klen - key0));   // valid keys (>= 1)
  const int my_key = 32 * q + n;               // lane's key within the tile
  const bool key_ok = my_key < nk;
  const int abs_key = key0 + my_key;           // for the causal test on self keys
  RowOffsets<D> ro0;
  ro0.init(n, G);
  RowOffsets<64> rt0;                          // transposed blocks: rows of 64 query slots
  rt0.init(n, G);

  // K and V of the workgroup's 128 keys, staged through the row buffers (64
  // keys per buffer), then held in registers as B fragments: K on P waves,
  // V on dS waves. Halves without keys are zero-filled.
  {
    const int sti = (int)st;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int nv = min(nk - 64 * h, 64);
      char *kd = h ? qr1 : qr0;
      char *vd = h ? or1 : or0;
      if (nv > 0) {
        const __bf16 *kb = kbase + (int64_t)(key0 + 64 * h) * st;
        const __bf16 *vb = vbase + (int64_t)(key0 + 64 * h) * st;
        dma_tile<D, 64, kNW>(kd, kb, [&](int r) { return r * sti; }, nv, wave, lane);
        dma_tile<D, 64, kNW>(vd, vb, [&](int r) { return r * sti; }, nv, wave, lane);
      } else {
        for (int i = tid; i < RB / 16; i += kFastThreads) {
          reinterpret_cast<u32x4 *>(kd)[i] = u32x4{0, 0, 0, 0};
          reinterpret_cast<u32x4 *>(vd)[i] = u32x4{0, 0, 0, 0};
        }
      }
    }
    wait_vmcnt<0>();
    lds_barrier();
  }

  const int qb_first = self ? (key0 * g) / QB : 0;
  const int nblk = __builtin_amdgcn_readfirstlane(nblk_all);

  // Block cursor: block blk of the workgroup's sequence is 64-row block
  // qb = qb_first + r of batch row b = uses[u] (the rows' block counts summed
  // over earlier uses give blk - r), with the element offsets of its rows
  // (GFAST), transposed block and statistics. Advancing within a batch row
  // adds constant strides; a new batch row (table loads) recomputes them.
  // Blocks past the end keep the last block's offsets and are not copied.
  // Every use has at least one block (rows without queries are not listed).
  struct Cursor {
    int blk, r, u, b, pu, nr, tok0;   // pu: blocks of this use; nr: packed rows of the row
    int64_t roff, rlim, toff, soff;   // rlim: bytes from roff to the group's last row
  };
  const int64_t row_step = (int64_t)(QB / g) * Hq * D;   // GFAST: elements between consecutive blocks
  auto use_row = [&](int u) __attribute__((always_inline)) {
    int b = self ? self_b : load_const(p.uses, __builtin_amdgcn_readfirstlane(use_b + u));
    // The table load is invariant, so the compiler could sink it (and its
    // latency) past a barrier into a matrix phase; this pins it here.
    asm volatile("" : "+s"(b));
    return b;
  };
  // Packed rows of batch row b (pinned like the use table load).
  auto row_geo = [&](int b, int &tok0, int &len, int &tblk0) __attribute__((always_inline)) {
    const DevRow rw = load_const(p.rows, b);
    tok0 = rw.tok0;
    len = rw.len;
    tblk0 = rw.tblk0;
    asm volatile("" : "+s"(tok0), "+s"(len), "+s"(tblk0));
  };
  auto cursor_set = [&](Cursor &c) __attribute__((always_inline)) {
    c.b = use_row(c.u);
    int tok0, len, tblk0;
    row_geo(c.b, tok0, len, tblk0);
    c.tok0 = tok0;
    c.nr = len * g;
    const int nqb = (c.nr + QB - 1) / QB;
    c.pu = nqb - qb_first;
    const int qb = qb_first + c.r;
    const int t0 = qb * (QB / g);                 // GFAST only
    c.roff = (((int64_t)tok0 + t0) * Hq + kvh * g) * D;
    // rows at or beyond the row's last packed row are positions >= len,
    // past the group's last row
    c.rlim = ((int64_t)(len - 1 - t0) * Hq + g) * D * 2;
    c.toff = ((int64_t)tblk0 + kvh * nqb + qb) * D * 64;
    c.soff = (int64_t)tok0 * Hq + kvh * c.nr + qb * QB;
  };
  auto cursor_at = [&](int blk) __attribute__((always_inline)) {
    Cursor c;
    c.blk = blk;
    int bl = min(blk, nblk - 1);
    c.u = 0;
    if (!self) {
      for (;;) {
        int tok0, len, tblk0;
        row_geo(use_row(c.u), tok0, len, tblk0);
        const int nb = (len * g + QB - 1) / QB;
        if (bl < nb) break;
        bl -= nb;
        ++c.u;
      }
    }
    c.r = bl;
    cursor_set(c);
    return c;
  };
  auto advance = [&](Cursor &c) __attribute__((always_inline)) {
    ++c.blk;
    if (c.blk < nblk) {
      if (++c.r == c.pu) {
        c.r = 0;
        ++c.u;
        cursor_set(c);
      } else {
        c.roff += row_step;
        c.rlim -= row_step * 2;
        c.toff += D * 64;
        c.soff += QB;
      }
    }
  };

  // --- copies of one block, by the four waves of one group ----------------
  // Packed row r0 + r of a block is query position (r0+r)/g, head (r0+r)%g of
  // the group. When g divides 64 (GFAST) every block starts on a position
  // boundary and a lane's element offset within the block is fixed.
  constexpr int CPI = D / 8;                   // 16-byte chunks per row
  constexpr int RPER = QB * CPI / 64 / 4;      // row-block copy instructions per wave
  int qfix[RPER];
#pragma unroll
  for (int i = 0; i < RPER; ++i) {
    const int pos = (q + 4 * i) * 64 + lane;
    const int r = pos / CPI;
    qfix[i] = ((r / g) * Hq + r % g) * D + ((pos % CPI) ^ swz<D>(r)) * 8;
  }
  CopyLanes<64, D, 4> ct;                      // transposed blocks: D rows of 64
  ct.init(q, lane);
  constexpr int TPER = CopyLanes<64, D, 4>::PER;
  static_assert(RPER * 8 == NMF, "one row-block copy per eight MFMAs");
  static_assert(32 % TPER == 0, "transposed-block copies spread over the 32 VALU elements");
  int tvoff[TPER];
#pragma unroll
  for (int i = 0; i < TPER; ++i) tvoff[i] = (ct.row[i] * 64 + ct.coff[i]) * 2;

  // A copy source: base address and resource size in bytes (0: nothing is
  // read, the copy writes zeros). Both are pinned when prepared, so their
  // scalar arithmetic stays in the VALU phase that prepares them; the buffer
  // resource is assembled at the copy.
  struct Src {
    const char *base;
    int bytes;
  };
  auto pin = [&](Src &x) __attribute__((always_inline)) { asm volatile("" : "+s"(x.base), "+s"(x.bytes)); };
  struct RowJob {
    Src s;
    int voff[RPER];
  };
  // Rows of the cursor's block of Q or dO.
  auto prep_rows = [&](const void *src, const Cursor &c) __attribute__((always_inline)) {
    RowJob jb;
    const bool live = c.blk < nblk;
    if constexpr (GFAST) {
      jb.s.base = (const char *)((const __bf16 *)src + c.roff);
      jb.s.bytes = live ? (int)min(c.rlim, (int64_t)0x7fffffff) : 0;
#pragma unroll
      for (int i = 0; i < RPER; ++i) jb.voff[i] = qfix[i] * 2;
    } else {
      const int r0 = (qb_first + c.r) * QB;
      const int nv = min(QB, c.nr - r0);
      const int t0 = r0 / g;
      const int64_t head0 = (((int64_t)c.tok0 + t0) * Hq + kvh * g) * D;
      // Packed row r is at element ((t - t0) Hq + h) D; rows at or beyond nv
      // lie outside the resource and read as zero.
      auto rowoff = [&](int r) __attribute__((always_inline)) {
        const int rr = r0 + r, t = rr / g;
        return ((t - t0) * Hq + (rr - t * g)) * D;
      };
      jb.s.base = (const char *)((const __bf16 *)src + head0);
      jb.s.bytes = live ? (rowoff(nv - 1) + D) * 2 : 0;
#pragma unroll
      for (int i = 0; i < RPER; ++i) {
        const int pos = (q + 4 * i) * 64 + lane;
        const int r = pos / CPI;
        jb.voff[i] = (rowoff(r) + ((pos % CPI) ^ swz<D>(r)) * 8) * 2;
      }
    }
    pin(jb.s);
    return jb;
  };
  auto issue_rows = [&](const RowJob &jb, int i, char *dst) __attribute__((always_inline)) {
    dma16(make_rsrc(jb.s.base, jb.s.bytes), jb.voff[i], dst + (q + 4 * i) * 1024);
  };
  // Transposed block of Q or dO.
  auto prep_t = [&](const void *src, const Cursor &c) __attribute__((always_inline)) {
    Src x{(const char *)((const __bf16 *)src + c.toff), c.blk < nblk ? D * 128 : 0};
    pin(x);
    return x;
  };
  auto issue_t = [&](const Src &x, int i, char *dst) __attribute__((always_inline)) {
    dma16(make_rsrc(x.base, x.bytes), tvoff[i], dst + (q + 4 * i) * 1024);
  };
  // LSE2 or D (64 floats; lanes at or beyond the row's packed rows read zero).
  auto prep_stat = [&](const float *src, const Cursor &c) __attribute__((always_inline)) {
    const int r0 = (qb_first + c.r) * QB;
    Src x{(const char *)(src + c.soff), c.blk < nblk ? min(QB, c.nr - r0) * 4 : 0};
    pin(x);
    return x;
  };
  auto issue_stat = [&](const Src &x, float *dst) __attribute__((always_inline)) {
    if (q == 0)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(make_rsrc(x.base, x.bytes), (lds_void_t *)dst, 4, lane * 4, 0, 0, 0);
  };

  // The two roles run separate code (PW: P wave); barriers pair up one to one.
  auto body = [&](auto PW) __attribute__((always_inline)) {
    constexpr bool pwave = decltype(PW)::value;
    // Lane offsets from this role's region (opaque to the compiler, so it
    // keeps one register per offset and folds each buffer into the immediate).
    constexpr int RBASE = pwave ? 0 : 4 * RB;
    RowOffsets<D> ro;
    RowOffsets<64> rt;
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      ro.off[s] = ro0.off[s] + RBASE;
      asm volatile("" : "+v"(ro.off[s]));
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      rt.off[s] = rt0.off[s] + RBASE;
      asm volatile("" : "+v"(rt.off[s]));
    }
    auto rel = [&](const char *buf) __attribute__((always_inline)) { return buf - RBASE; };
    bf16x8 kv[NSTEP];
    {
      const char *src = pwave ? ((q >> 1) ? qr1 : qr0) : ((q >> 1) ? or1 : or0);
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) kv[s] = row_frag_at<D>(rel(src), ro, 32 * (q & 1), s);
      lds_barrier();
    }
    f32x16 acc[DT];                              // dV^T (P waves) or dK^T (dS waves): [channel][key]
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = zero16();
    f32x16 sp[2];                                // S (P waves) or dP (dS waves) of both 32-row subtiles
    bf16x8 pk[4];                                // P (P waves) or dS (dS waves), k-step 2 sub + h

    // -D of a block's rows crow(j, G) of both subtiles, straight into the dP
    // accumulators: register 4k + e of subtile sub is row 32 sub + 8k + 4G + e.
    auto init_nd = [&](const float *ndn) __attribute__((always_inline)) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const f32x4 v = *reinterpret_cast<const f32x4 *>(ndn + 32 * sub + 8 * k + 4 * G);
#pragma unroll
          for (int e = 0; e < 4; ++e) sp[sub][4 * k + e] = v[e];
        }
    };
    // Matrix phase: 2 NSTEP MFMAs on row fragments of `rows` (S or dP of the
    // next block) and 2 NSTEP on transposed fragments of `tr` times pk (dV or
    // dK of this block); TR_FIRST puts the transposed product first. One LDS
    // fragment per MFMA, LEAD fragments ahead; row-block copy piece n after
    // MFMA 8n + 7. With TR_FIRST (dS wave) the dP accumulator starts at -D of
    // the next block (ndn), so the MFMAs deliver dP - D.
    auto matrix = [&](auto TR_FIRST, const char *rows, const char *tr, const float *ndn, auto &&piece)
                      __attribute__((always_inline)) {
      constexpr bool TF = decltype(TR_FIRST)::value;
      constexpr int H = 2 * NSTEP;
      auto frag = [&](auto K) __attribute__((always_inline)) {
        constexpr int k = decltype(K)::value;
        constexpr bool is_tr = TF ? (k < H) : (k >= H);
        constexpr int kk = TF ? (k < H ? k : k - H) : (k < H ? k : k - H);
        if constexpr (is_tr) return row_frag_at<64>(tr, rt, 32 * (kk / 4), kk % 4);
        else return row_frag_at<D>(rows, ro, 32 * (kk / NSTEP), kk % NSTEP);
      };
      if constexpr (TF) init_nd(ndn);
      else {
        sp[0] = zero16();
        sp[1] = zero16();
      }
      // The SIMD's other wave is in its VALU phase: let this wave's MFMA
      // stream issue first.
      __builtin_amdgcn_s_setprio(PRIO);
      bf16x8 ring[RING];
      static_for<LEAD>([&](auto K) __attribute__((always_inline)) { ring[decltype(K)::value] = frag(K); });
      static_for<NMF>([&](auto K) __attribute__((always_inline)) {
        constexpr int k = decltype(K)::value;
        constexpr bool is_tr = TF ? (k < H) : (k >= H);
        constexpr int kk = k < H ? k : k - H;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (k + LEAD < NMF) ring[(k + LEAD) % RING] = frag(std::integral_constant<int, k + LEAD>{});
        if constexpr (is_tr) acc[kk / 4] = Mma<__bf16>::run(ring[k % RING], pk[kk % 4], acc[kk / 4]);
        else sp[kk / NSTEP] = Mma<__bf16>::run(ring[k % RING], kv[kk % NSTEP], sp[kk / NSTEP]);
        if constexpr ((k & 7) == 7) piece(k >> 3);
      });
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
    };
    // S or dP - D of block 0 alone (prologue).
    auto first_rows = [&](const char *rows, const float *ndn) __attribute__((always_inline)) {
      if constexpr (pwave) {
        sp[0] = zero16();
        sp[1] = zero16();
      } else {
        init_nd(ndn);
      }
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) {
        sp[0] = Mma<__bf16>::run(row_frag_at<D>(rows, ro, 0, s), kv[s], sp[0]);
        sp[1] = Mma<__bf16>::run(row_frag_at<D>(rows, ro, 32, s), kv[s], sp[1]);
      }
    };
    char *const xme = xch + q * 4096 + lane * 16;   // this lane's P slots (4 x 16 bytes, 1 KiB apart)

    // P wave VALU phase: P of block blk from sp (S) and its LSE2 in lsb; packed
    // into pk and published to the SIMD's dS wave. piece(n) issues copy
    // instruction n, spread over the elements.
    auto p_valu = [&](auto CAUSAL, int blk, const float *lsb, auto &&piece) __attribute__((always_inline)) {
      constexpr bool CA = decltype(CAUSAL)::value;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        int lo = 0;
        if constexpr (CA) {
          // self tiles have a single use: block blk is 64-row block qb_first + blk
          lo = abs_key * g - ((qb_first + blk) * QB + 32 * sub) - 4 * G;   // rows at or after the key's position
        }
        f32x4 lsv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) lsv[k] = *reinterpret_cast<const f32x4 *>(lsb + 32 * sub + 8 * k + 4 * G);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          float pv = fast_exp2(fmaf(sp[sub][j], c, -lsv[j >> 2][j & 3]));
          if constexpr (CA) pv = crow(j, 0) >= lo ? pv : 0.0f;
          sp[sub][j] = pv;
          constexpr int EPP = 32 / TPER;     // elements per copy piece
          if ((16 * sub + j) % EPP == EPP - 1) piece((16 * sub + j) / EPP);
        }
        pk[2 * sub] = pack_bf16x8(sp[sub], 0);
        pk[2 * sub + 1] = pack_bf16x8(sp[sub], 1);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) *reinterpret_cast<bf16x8 *>(xme + t * 1024) = pk[t];
      fence_regs(pk);
    };
    // dS wave VALU phase: dS = P (dP - D) of a block from the published P and
    // sp (dP - D); piece(n) as for the P wave.
    auto ds_valu = [&](auto &&piece) __attribute__((always_inline)) {
      bf16x8 pv[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) pv[t] = *reinterpret_cast<const bf16x8 *>(xme + t * 1024);
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          sp[sub][j] = (float)pv[2 * sub + (j >> 3)][j & 7] * sp[sub][j];
          constexpr int EPP = 32 / TPER;
          if ((16 * sub + j) % EPP == EPP - 1) piece((16 * sub + j) / EPP);
        }
        pk[2 * sub] = pack_bf16x8(sp[sub], 0);
        pk[2 * sub + 1] = pack_bf16x8(sp[sub], 1);
      }
      fence_regs(pk);
    };

    // One wave's copy batch: rows of a block of Q or dO, a transposed block,
    // one statistics block (wave q == 0 of the group).
    struct Batch {
      RowJob rows;
      Src tr, stat;
    };
    // Batch prepared one VALU phase ahead: rows (and the P wave's LSE2) of
    // block `hi`, the transposed block (and the dS wave's D) of block hi - 1.
    // The two cursors advance by one block per step.
    Batch nb;
    Cursor chi, clo;                             // set once nblk > 0 is known
    auto prep = [&]() __attribute__((always_inline)) {
      if constexpr (pwave) {
        nb.rows = prep_rows(p.d_o, chi);
        nb.tr = prep_t(p.qT, clo);
        nb.stat = prep_stat(p.lse2, chi);
      } else {
        nb.rows = prep_rows(p.q, chi);
        nb.tr = prep_t(p.doT, clo);
        nb.stat = prep_stat(p.nd, chi);
      }
      advance(chi);
      advance(clo);
    };
    auto rows_piece = [&](char *dst) __attribute__((always_inline)) {
      return [&nb, dst, &issue_rows](int n) __attribute__((always_inline)) { issue_rows(nb.rows, n, dst); };
    };
    auto tr_piece = [&](const Batch &bt, char *tdst, float *sdst) __attribute__((always_inline)) {
      return [&bt, tdst, sdst, &issue_t, &issue_stat](int n) __attribute__((always_inline)) {
        issue_t(bt.tr, n, tdst);
        if (n == 0) issue_stat(bt.stat, sdst);
      };
    };

    // A wave's batch is split: its row-block copies go into a matrix phase (one
    // per eight MFMAs), its transposed-block and statistics copies into a VALU
    // phase, so no phase issues more than a few copies and the copy queue
    // never stalls the issuing wave for long. At the end of each matrix phase
    // a wave waits for everything but that phase's row copies.
    //
    // P wave, block i (batch i: dO rows of i+2, Q^T_{i+1}, LSE2 of i+2).
    // A_i: S_{i+1} from rows of i+1 (qrn), dV from dO^T_i (ot); dO rows of
    // i+2 into orw. B_i: P_{i+1} with LSE2 of i+1 (lsn); Q^T_{i+1} into qtw,
    // LSE2 of i+2 into lsw; then batch i+1 is prepared.
    auto p_step = [&](auto CAUSAL, int i, const char *qrn, const char *ot, char *orw, char *qtw, float *lsw,
                      const float *lsn) __attribute__((always_inline)) {
      matrix(std::false_type{}, rel(qrn), rel(ot), nullptr, rows_piece(orw));
      wait_vmcnt<RPER>();                        // batch i-1 has landed
      lds_barrier();
      const Batch cur = nb;
      p_valu(CAUSAL, i + 1, lsn, tr_piece(cur, qtw, lsw));
      prep();
      lds_barrier();                             // also waits for any table load
    };
    // dS wave, block i (batch i: Q rows of i+2, dO^T_{i+1}, -D of i+2; its
    // rows were copied during B_{i-1}). A_i: dS_i; dO^T_{i+1} into otw, -D of
    // i+2 into ndw; then batch i+1 is prepared. B_i: dK from Q^T_i (qt),
    // dP_{i+1} - D from dO rows of i+1 (orn) and -D of i+1 (ndn); Q rows of
    // i+3 into qrw.
    auto ds_step = [&](int i, const float *ndn, const char *qt, const char *orn, char *qrw, char *otw,
                       float *ndw) __attribute__((always_inline)) {
      const Batch cur = nb;
      ds_valu(tr_piece(cur, otw, ndw));
      prep();
      lds_barrier();                             // also waits for any table load
      matrix(std::true_type{}, rel(orn), rel(qt), ndn, rows_piece(qrw));
      wait_vmcnt<RPER>();                        // batch i has landed
      lds_barrier();
    };

    if (nblk > 0) {
      chi = cursor_at(2);
      clo = cursor_at(1);
      // Blocks 0 and 1: rows of 0 and 1, Q^T_0 / dO^T_0, LSE2 and -D of 0 and 1.
      if constexpr (pwave) {
        const Cursor c0 = cursor_at(0);
        RowJob rj = prep_rows(p.q, c0);
#pragma unroll
        for (int k = 0; k < RPER; ++k) issue_rows(rj, k, qr0);
        rj = prep_rows(p.q, clo);
#pragma unroll
        for (int k = 0; k < RPER; ++k) issue_rows(rj, k, qr1);
        const Src tj = prep_t(p.qT, c0);
#pragma unroll
        for (int k = 0; k < TPER; ++k) issue_t(tj, k, qt0);
        issue_stat(prep_stat(p.lse2, c0), ls0);
        issue_stat(prep_stat(p.lse2, clo), ls1);
      } else {
        const Cursor c0 = cursor_at(0);
        RowJob rj = prep_rows(p.d_o, c0);
#pragma unroll
        for (int k = 0; k < RPER; ++k) issue_rows(rj, k, or0);
        rj = prep_rows(p.d_o, clo);
#pragma unroll
        for (int k = 0; k < RPER; ++k) issue_rows(rj, k, or1);
        const Src tj = prep_t(p.doT, c0);
#pragma unroll
        for (int k = 0; k < TPER; ++k) issue_t(tj, k, ot0);
        issue_stat(prep_stat(p.nd, c0), dv0);
        issue_stat(prep_stat(p.nd, clo), dv1);
      }
      wait_vmcnt<0>();
      lds_barrier();
      if constexpr (pwave) {
        auto run = [&](auto CAUSAL) __attribute__((always_inline)) {
          // Distinct markers keep the compiler from hoisting the two variants'
          // common first loads above the branch (they would stay live across
          // the other variant's loop).
          if constexpr (decltype(CAUSAL)::value) asm volatile("; causal tiles" ::: "memory");
          else asm volatile("; prefix tiles" ::: "memory");
          first_rows(rel(qr0), nullptr);
          p_valu(CAUSAL, 0, ls0, [](int) {});
          prep();                                // batch 0
          lds_barrier();
          for (int i = 0; i < nblk; i += 2) {
            p_step(CAUSAL, i, qr1, ot0, or0, qt1, ls0, ls1);
            if (i + 1 >= nblk) break;
            p_step(CAUSAL, i + 1, qr0, ot1, or1, qt0, ls1, ls0);
          }
        };
        if (self) run(std::true_type{});
        else run(std::false_type{});
      } else {
        first_rows(rel(or0), dv0);
        prep();                                  // batch 0
        lds_barrier();
        {
          auto rp = rows_piece(qr0);             // batch 0's rows (Q rows of 2)
#pragma unroll
          for (int k = 0; k < RPER; ++k) rp(k);
        }
        for (int i = 0; i < nblk; i += 2) {
          ds_step(i, dv1, qt0, or1, qr1, ot1, dv0);
          if (i + 1 >= nblk) break;
          ds_step(i + 1, dv0, qt1, or0, qr0, ot0, dv1);
        }
      }
      wait_vmcnt<0>();
    }

    // Store through LDS: each lane holds 4-channel pieces of its key's row;
    // staged as whole rows, every store instruction writes full 16-byte
    // pieces of consecutive rows (whole cache lines instead of 8-byte pieces
    // that leave lines partly written). Every wave's copies have landed
    // (wait above), so after this barrier the arena is free.
    __syncthreads();
    __bf16 *dst = pwave ? dvp : dkp;
    if (!dst) return;
    const float sc = pwave ? 1.0f : p.scale;
    constexpr int SRS = (D + 8) * 2;                 // staged row bytes (padded against bank conflicts)
    char *const stg = smem + wave * 32 * SRS;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        store4(reinterpret_cast<__bf16 *>(stg + n * SRS) + dt * 32 + jj * 8 + G * 4, acc[dt][jj * 4 + 0] * sc,
               acc[dt][jj * 4 + 1] * sc, acc[dt][jj * 4 + 2] * sc, acc[dt][jj * 4 + 3] * sc);
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's LDS writes are done
    asm volatile("" ::: "memory");
    constexpr int CPR = D / 8;                       // 16-byte pieces per row
    constexpr int RPI = 64 / CPR;                    // rows per store instruction
    const int nrow = min(32, nk - 32 * q);           // valid keys of this wave
    const int pr = lane / CPR, pc = lane % CPR;
#pragma unroll
    for (int i = 0; i < 32 / RPI; ++i) {
      const int r = RPI * i + pr;
      const uint4 v = *reinterpret_cast<const uint4 *>(stg + r * SRS + pc * 16);
      if (r < nrow) *reinterpret_cast<uint4 *>(dst + (int64_t)(key0 + 32 * q + r) * st + pc * 8) = v;
    }

  };
  if (pwave) body(std::true_type{});
  else body(std::false_type{});
}

hipError_t launch_fwd_bf16(const FwdParams &p, int D, hipStream_t s) {
  const int64_t grid = p.n_items;
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
  const int64_t grid = p.n_items;
  if (D == 64)
    hipLaunchKernelGGL(dq_bf16_kernel<64>, dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
  else
    hipLaunchKernelGGL(dq_bf16_kernel<128>, dim3((unsigned)grid), dim3(kFastThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_dkdv_bf16(const DkdvParams &p, int D, int n_wg, hipStream_t s) {
  const dim3 grid((unsigned)n_wg);
  const bool gfast = kDkdvQBlock % p.g == 0;
  if (D == 64) {
    if (gfast) hipLaunchKernelGGL((dkdv_bf16_kernel<64, true>), grid, dim3(kFastThreads), 0, s, p);
    else hipLaunchKernelGGL((dkdv_bf16_kernel<64, false>), grid, dim3(kFastThreads), 0, s, p);
  } else {
    if (gfast) hipLaunchKernelGGL((dkdv_bf16_kernel<128, true>), grid, dim3(kFastThreads), 0, s, p);
    else hipLaunchKernelGGL((dkdv_bf16_kernel<128, false>), grid, dim3(kFastThreads), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_prologue_bf16(const PreParams &p, int D, hipStream_t s) {
  const dim3 grid((unsigned)(p.Hkv * p.nqb_max), (unsigned)p.B);
  if (D == 64)
    hipLaunchKernelGGL(bwd_prologue_bf16_kernel<64>, grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(bwd_prologue_bf16_kernel<128>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace cas
