// Internal layouts shared by the libcas host planner and its HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cas.h"

namespace cas {

// Work decomposition (gfx950: 64-lane waves, 4 SIMDs per CU).
constexpr int kThreads = 256;       // 4 waves per workgroup
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerWave = 64;    // packed query rows a wave owns in fwd / dQ
constexpr int kRowsPerWg = kRowsPerWave * kWaves;   // 256
constexpr int kDqRowsPerWave = 32;  // dQ holds Q, dO and the dQ sums in registers
constexpr int kDqRowsPerWg = kDqRowsPerWave * kWaves;  // 128
constexpr int kKeyTile = 64;        // keys per LDS tile in fwd / dQ
constexpr int kDkdvKeysPerWave = 32;
constexpr int kDkdvKeyTile = kDkdvKeysPerWave * kWaves;  // 128 keys per dK/dV workgroup
constexpr int kDkdvQBlock = 64;     // query rows per LDS block in dK/dV
constexpr int kMaxSplits = 32;

// A "packed row" r of (batch b, kv head kvh) is query position t = r / g of
// query head kvh*g + r % g: the g heads of one position are adjacent rows, so
// one K/V tile in LDS serves the whole GQA group.

// Prefix entry of one batch row (forward and dQ walks).
struct DevSeg {
  const void *k;
  const void *v;
  int64_t stride_tok;
  int64_t stride_head;
  int32_t len;
  int32_t tile_begin;   // first kKeyTile tile of this entry within the row's prefix
};

// One batch row (a sample). Its query tokens are tokens tok0 .. tok0+len-1
// of the token axis of q, o, d_o, dq and the self K/V (row b of a fixed-length
// batch starts at b * q_len; packed samples start where the previous one
// ends). Per-row statistics (-D, LSE2, split partials) of KV head kvh and
// packed row r sit at tok0 * Hq + kvh * len * g + r.
struct DevRow {
  int32_t seg_begin;
  int32_t seg_end;
  int32_t prefix_tiles;  // kKeyTile tiles over the row's whole prefix
  int32_t tile_begin;    // the row's first entry in the DevTile table
  int32_t tok0;          // first query token of the row
  int32_t len;           // query tokens of the row (>= 0)
  int32_t lse0;          // lse index of (head 0, position 0); head h adds h * lse_hs
  int32_t tblk0;         // bf16 backward: first transposed 64-row block of the row
};

// One kKeyTile-key tile of a row's prefix (bf16 forward and dQ): its first key
// at KV head 0 and the strides to reach the other heads and keys.
struct DevTile {
  const void *k;
  const void *v;
  int64_t stride_head;
  int32_t stride_tok;
  int32_t nvalid;        // keys in the tile, 1 .. kKeyTile
};

// Distinct cartridge after alias folding (dK/dV pass).
struct DevCart {
  const void *k;
  const void *v;
  void *dk;
  void *dv;
  int64_t stride_tok;
  int64_t stride_head;
  int32_t len;
  int32_t tile_begin;   // first kDkdvKeyTile tile in the dK/dV grid
  int32_t use_begin;    // uses[use_begin .. use_end) = batch rows referencing it
  int32_t use_end;
  int32_t nblk;         // 64-row query blocks over all uses (sum of the rows' block counts)
  int32_t pad_;
};

// One dK/dV workgroup: a key tile (cartridge tiles first, then self tile
// j of batch row b as cart_tiles + b * self_tiles + j) and a KV head. The host
// lists them longest first (most query blocks), so the long workgroups of
// every KV head start in the first wave of the dispatch.
struct DevWg {
  int32_t tile;
  int32_t kvh;
};

// The bf16 dK/dV list of one XCD: entries [off, off + cnt) of the order table.
// Workgroup j of the XCD takes entry off + j while j < head; the entries from
// head on (the list's shortest) are claimed at run time, first by the XCD's
// own workgroups, then by any XCD that has run out of its own.
struct DevQueue {
  int32_t off;
  int32_t cnt;
  int32_t head;
  int32_t pad;
};

// One workgroup of the bf16 forward or dQ kernel: 256-row query block qblk
// of batch row b at KV head kvh, key-axis split `split`.
struct DevItem {
  int32_t qblk;
  int32_t split;
  int32_t b;
  int32_t kvh;
};

enum DType : int32_t { kBF16 = 0, kFP32 = 1 };

struct FwdParams {
  const void *q;
  const void *k_self;
  const void *v_self;
  void *o;
  float *lse;
  float *part_o;      // [splits][plane][D] when splits > 1 (rows as the statistics)
  float *part_lse;    // [splits][plane]
  const DevSeg *segs;
  const DevRow *rows;
  const DevTile *tiles;
  const DevItem *items;       // [n_items] bf16: workgroup i takes items[i]
  int32_t *ovf_flag;  // [grid] bf16: workgroup needs the exact-maximum pass
  int64_t plane;      // T * Hq: rows of one split partial plane
  int32_t B, Smax, Hkv, g, nrows_max, nqblk, splits;
  int32_t lse_hs;     // lse head stride (q_len, or T for packed samples)
  int32_t n_items;    // bf16 grid
  float scale_log2;   // softmax_scale * log2(e)
};

struct MergeParams {
  const float *part_o;
  const float *part_lse;
  void *o;
  float *lse;
  const DevRow *rows;
  int64_t plane;
  int32_t B, Hkv, g, nrows_max, splits, lse_hs;
};

struct PreParams {
  const void *o;
  const void *d_o;
  const float *lse;
  float *nd;     // per-row statistics (see DevRow): -rowsum(dO * O)  (D negated)
  float *lse2;   // LSE * log2(e)
  const void *q;
  void *qT;      // bf16: per row, [Hkv][nqb][D][64] Q of each 64-row block, transposed
  void *doT;     // bf16: same for dO
  const DevRow *rows;
  int32_t B, Hkv, g, nrows_max, nqb_max, lse_hs;
};

struct DqParams {
  const void *q;
  const void *k_self;
  const void *v_self;
  const void *d_o;
  const float *nd;        // -D
  const float *lse2;
  void *dq;
  float *part_dq;   // [splits][plane][D] when splits > 1 (rows as the statistics)
  const DevSeg *segs;
  const DevRow *rows;
  const DevTile *tiles;
  const DevItem *items;       // [n_items] bf16: workgroup i takes items[i]
  int64_t plane;
  int32_t B, Smax, Hkv, g, nrows_max, nqblk, splits;
  int32_t n_items;    // bf16 grid
  float scale_log2;
  float scale;
};

struct DqReduceParams {
  const float *part_dq;
  void *dq;
  const DevRow *rows;
  int64_t plane;
  int32_t B, Hkv, g, nrows_max, splits;
  float scale;
};

struct DkdvParams {
  const void *q;
  const void *k_self;
  const void *v_self;
  const void *d_o;
  const float *nd;        // -D
  const float *lse2;
  const void *qT;           // bf16: transposed Q / dO blocks (see PreParams)
  const void *doT;
  void *dk_self;
  void *dv_self;
  const DevCart *carts;
  const int32_t *uses;
  const DevRow *rows;
  const DevWg *order;       // the workgroups' tiles and KV heads ([grid] without queues)
  const DevQueue *queues;   // bf16: [xcds] per-XCD lists of `order`, or null (entry = workgroup id)
  int32_t *claim;           // bf16: [xcds] tail entries claimed so far (zero at launch)
  int32_t xcds;             // bf16 with queues: workgroup i runs on XCD i % xcds
  int32_t n_carts;
  int32_t cart_tiles;       // dK/dV tiles over all distinct cartridges
  int32_t self_tiles;       // dK/dV tiles per batch row over the self keys (longest row)
  int32_t B, Hkv, g;
  float scale_log2;
  float scale;
};

// Cartridge Adam step: one trainable tensor (a cartridge's K or V).
struct DevAdamT {
  __bf16 *x;             // parameters (strided like the segment)
  const __bf16 *g;       // gradient, same strides
  float *m1;             // moments, contiguous [len][Hkv][d]
  float *m2;
  int64_t stride_tok;
  int64_t stride_head;
  int32_t len;
  int32_t frozen;        // leading tokens left untouched
  float lr;              // lr * warmup factor
  float bc1, bc2;        // 1 - beta^t, rounded to fp32
  int32_t pad_[3];
};

// One workgroup's share: kAdamChunk tokens of tensor `t` from token `tok0`.
struct DevAdamChunk {
  int32_t t;
  int32_t tok0;
};
constexpr int kAdamChunk = 16;

struct AdamParams {
  const DevAdamT *tensors;
  const DevAdamChunk *chunks;
  int32_t Hkv;
  float beta1, beta2, omb1, omb2;   // omb = 1 - beta (fp32)
  float eps;
};

// Paged decode: one request (its queries are tokens q0 .. q0+n-1; its keys
// the pages page_ids[page0 ..] in order, kv_len of them) and one workgroup's
// share: packed rows row0 .. row0+15 (row r = query r / g, head kvh*g + r % g)
// over 32-key tiles [tile0, tile1) of the request's key axis.
constexpr int kDecTile = 32;
constexpr int kDecRows = 16;
struct DevDecodeReq {
  int32_t q0, n, kv_len, page0;
  int32_t nsplit;        // key-axis splits of every row block of the request
  int32_t pad_[3];
};
struct DevDecodeWork {
  int32_t b, kvh, row0, split;   // split index, or -1 when the range is the whole axis
  int32_t tile0, tile1;
  int32_t pad_[2];
};

struct DecodeParams {
  const void *q;
  const void *k_pages;
  const void *v_pages;
  void *o;
  float *lse;             // [Hq][Tq] or null
  const DevDecodeReq *reqs;
  const DevDecodeWork *work;
  const int32_t *page_ids;
  const int32_t *tok_req; // [Tq] request of each query token (merge)
  float *part_o;          // [split][Tq * Hq][D] when a request is split
  float *part_lse;        // [split][Tq * Hq]
  int64_t plane;          // Tq * Hq
  int32_t Hkv, g, page_size, Tq;
  float scale_log2;
};

// Forward shared by cas_prefix_attn_fwd (scratch == nullptr: the caller's
// workspace, tables through the pinned staging ring) and the no-allocation
// forward (scratch != nullptr: after validation, scratch() yields the device
// address of the library's static scratch of ws_bytes; the forward's key
// splits are lowered until its workspace fits, tables go up as kernel
// arguments, and no timing events are recorded).
using ScratchAddressFn = hipError_t (*)(void **);
cas_status_t prefix_attn_fwd_run(const cas_problem_t *p, const void *q, const void *k_self,
                                 const void *v_self, void *o, float *lse, void *workspace,
                                 size_t ws_bytes, hipStream_t stream, ScratchAddressFn scratch);

// Copies `bytes` (a multiple of 16) of host memory to device memory `dst` on
// stream s as the kernel arguments of a copy kernel, kTableArgChunk bytes per
// launch: no host or device allocation.
constexpr int kTableArgChunk = 2048;
hipError_t launch_table_args_upload(const void *host, size_t bytes, void *dst, hipStream_t s);

// Kernel launchers (defined in the .hip files).
hipError_t launch_fwd(const FwdParams &p, DType dt, int D, hipStream_t s);
hipError_t launch_fwd_merge(const MergeParams &p, DType dt, int D, hipStream_t s);
// Copies `bytes` of pinned host memory to device memory (both 16-byte
// aligned) with a kernel on stream s.
hipError_t launch_table_upload(void *dst, const void *src, size_t bytes, hipStream_t s);
hipError_t launch_bwd_pre(const PreParams &p, DType dt, int D, hipStream_t s);
hipError_t launch_dq(const DqParams &p, DType dt, int D, hipStream_t s);
hipError_t launch_dq_reduce(const DqReduceParams &p, DType dt, int D, hipStream_t s);
hipError_t launch_dkdv(const DkdvParams &p, DType dt, int D, int n_wg, hipStream_t s);
// bf16 fast path (8-wave workgroups; forward and dQ take 256 packed rows per workgroup).
constexpr int kBf16RowsPerWg = 256;
hipError_t launch_fwd_bf16(const FwdParams &p, int D, hipStream_t s);
hipError_t launch_dq_bf16(const DqParams &p, int D, hipStream_t s);
hipError_t launch_dkdv_bf16(const DkdvParams &p, int D, int n_wg, hipStream_t s);
hipError_t launch_bwd_prologue_bf16(const PreParams &p, int D, hipStream_t s);
hipError_t launch_adam_bf16(const AdamParams &p, int D, int n_chunks, hipStream_t s);
hipError_t launch_decode_bf16(const DecodeParams &p, int D, int n_work, hipStream_t s);
hipError_t launch_decode_merge_bf16(const DecodeParams &p, int D, hipStream_t s);

}  // namespace cas
