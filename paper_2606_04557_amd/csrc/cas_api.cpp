// libcas host side: argument validation, launch planning, segment-table
// upload, kernel launches, cartridge staging and optional kernel timing.
//
// Validation is pure host code and runs before any HIP call, so every error
// path can be exercised on a machine without a GPU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/cas.h"
#include "cas_host.h"
#include "cas_internal.h"

using namespace cas;

namespace {

thread_local std::string g_err;

cas_status_t fail(cas_status_t s, const std::string &msg) {
  g_err = msg;
  return s;
}

std::mutex g_tuning_mu;
cas_tuning_t g_tuning = {0, 0};

cas_tuning_t tuning() {
  std::lock_guard<std::mutex> lk(g_tuning_mu);
  return g_tuning;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

struct Interval {
  uintptr_t lo, hi;   // [lo, hi)
  bool write;
  uintptr_t owner;    // identical writes of one owner may coincide (aliased cartridge)
  const char *what;
};

// Every write interval must be disjoint from every other interval (reads and
// writes) of a different owner.
bool overlap_free(std::vector<Interval> &iv, std::string &msg) {
  std::sort(iv.begin(), iv.end(), [](const Interval &a, const Interval &b) { return a.lo < b.lo; });
  uintptr_t max_hi_any = 0, max_hi_wr = 0;
  int any_idx = -1, wr_idx = -1;
  for (size_t i = 0; i < iv.size(); ++i) {
    const Interval &x = iv[i];
    if (x.hi <= x.lo) continue;
    if (x.write && any_idx >= 0 && max_hi_any > x.lo &&
        !(iv[any_idx].write && iv[any_idx].owner == x.owner && iv[any_idx].lo == x.lo &&
          iv[any_idx].hi == x.hi)) {
      msg = std::string("output ") + x.what + " overlaps " + iv[any_idx].what;
      return false;
    }
    if (!x.write && wr_idx >= 0 && max_hi_wr > x.lo) {
      msg = std::string("input ") + x.what + " overlaps output " + iv[wr_idx].what;
      return false;
    }
    if (x.hi > max_hi_any) {
      max_hi_any = x.hi;
      any_idx = (int)i;
    }
    if (x.write && x.hi > max_hi_wr) {
      max_hi_wr = x.hi;
      wr_idx = (int)i;
    }
  }
  return true;
}

struct Plan {
  DType dt;
  int esize;
  int B, Hkv, g, Hq, D;
  bool packed = false;
  int Sq = 0;              // fixed-length rows: q_len
  int64_t T = 0;           // tokens over all rows
  int Smax = 0;            // longest row
  int nrows_max = 0;       // Smax * g
  int nqb_max = 0;         // 64-row blocks of the longest row
  std::vector<int32_t> tok0, len;
  float scale;
  std::vector<DevSeg> segs;
  std::vector<DevRow> rows;
  std::vector<DevTile> tiles;
  std::vector<DevItem> items;       // bf16 forward (or, backward plan, dQ) workgroups in dispatch order
  std::vector<DevCart> carts;
  std::vector<int32_t> uses;
  std::vector<DevWg> order;       // dK/dV workgroups, longest first
  std::vector<DevQueue> queues;   // bf16 dK/dV: per-XCD lists of `order` (empty: entry = workgroup id)
  int64_t dkdv_grid = 0;          // dK/dV workgroups launched
  int self_tiles_max = 0;         // dK/dV self tiles of the longest row
  int64_t order_cap = 0;          // order entries with every self tile
  int64_t max_prefix = 0;
  int fwd_splits = 1, dq_splits = 1;
  int xcds = 8;                   // XCDs of the device (workgroup order of the bf16 kernels)
  int cus = 256;                  // compute units of the device
  int nqblk_fwd = 0, nqblk_dq = 0;
  int cart_tiles = 0;
  bool want_self_grad = false;
  // workspace layout
  size_t off_segs = 0, off_rows = 0, off_tiles = 0, off_items = 0, off_carts = 0, off_uses = 0, off_order = 0,
         off_queues = 0, off_claim = 0,
         table_bytes = 0;
  size_t off_part_o = 0, off_part_lse = 0, off_ovf = 0, ws_fwd = 0;
  size_t off_nd = 0, off_lse2 = 0, off_part_dq = 0, off_qT = 0, off_doT = 0, ws_bwd = 0;
};

// Compute units and XCDs of the current device, looked up once per device.
// gfx950 has 32 CUs per XCD (256 and 8 on a whole MI355X; a partition shows
// fewer). Without a device (planning-only use) the whole MI355X is assumed.
struct Topology {
  int cus = 256, xcds = 8;
};
std::mutex g_topo_mu;
std::map<int, Topology> g_topo;
Topology device_topology() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return Topology{};
  }
  std::lock_guard<std::mutex> lk(g_topo_mu);
  auto it = g_topo.find(dev);
  if (it != g_topo.end()) return it->second;
  Topology t;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0) {
    t.cus = cus;
    t.xcds = std::max(1, cus / 32);
  } else {
    (void)hipGetLastError();
  }
  g_topo.emplace(dev, t);
  return t;
}

// Key-axis splits for a grid of base_wgs workgroups: aim at two workgroups
// per compute unit.
int auto_splits(int64_t base_wgs, int64_t min_row_tiles, int cus) {
  const int64_t target = 2 * (int64_t)cus;
  if (base_wgs >= (target * 3) / 4) return 1;
  int64_t s = ceil_div(target, std::max<int64_t>(1, base_wgs));
  s = std::min<int64_t>(s, std::max<int64_t>(1, min_row_tiles / 8));
  return (int)std::max<int64_t>(1, std::min<int64_t>(s, kMaxSplits));
}

// Workgroups of the bf16 forward and dQ kernels, in dispatch order, with
// `splits` key-axis splits. Workgroup i is dispatched to XCD i mod X (X = 8 on
// a whole MI355X, each XCD with its own L2), and each XCD hands its next
// workgroup to whichever of its CUs frees first. The items are enumerated
// KV head slowest, then batch row (most key tiles first), split, query block,
// and cut into X contiguous shares, share x for XCD x: the workgroups that
// stream one (row, KV head)'s K/V tiles share an L2 and, when X divides the
// KV heads, every XCD gets whole KV heads (the same work). Within a share the
// items go longest first (key tiles walked; ties keep the enumeration
// order): with one workgroup per CU at a time that is the
// longest-processing-time rule, so the shortest start last and the CUs
// finish together. Only query blocks that hold rows are listed.
void build_items(Plan &pl, int splits) {
  std::vector<int> rows(pl.B);
  for (int b = 0; b < pl.B; ++b) rows[b] = b;
  std::stable_sort(rows.begin(), rows.end(), [&](int a, int c) {
    return pl.rows[a].prefix_tiles + ceil_div(pl.len[a], kKeyTile) >
           pl.rows[c].prefix_tiles + ceil_div(pl.len[c], kKeyTile);
  });
  struct E {
    DevItem it;
    int64_t tiles;
  };
  std::vector<E> v;
  for (int kvh = 0; kvh < pl.Hkv; ++kvh)
    for (int b : rows) {
      const int64_t nrows = (int64_t)pl.len[b] * pl.g;
      const int nq = (int)ceil_div(nrows, kBf16RowsPerWg);
      for (int sp = 0; sp < splits; ++sp)
        for (int qb = nq - 1; qb >= 0; --qb) {
          // The kernels' tile range: the prefix, then the self tiles up to
          // the block's last query position, cut evenly over the splits.
          const int64_t r1 = std::min<int64_t>(nrows, (int64_t)(qb + 1) * kBf16RowsPerWg);
          const int64_t nt = pl.rows[b].prefix_tiles + ((r1 - 1) / pl.g) / kKeyTile + 1;
          v.push_back({{qb, sp, b, kvh}, nt * (sp + 1) / splits - nt * sp / splits});
        }
    }
  const size_t n = v.size(), X = (size_t)std::max(1, pl.xcds), per = n / X;
  auto sort_share = [&](size_t lo, size_t hi) {
    std::stable_sort(v.begin() + lo, v.begin() + hi, [](const E &a, const E &c) { return a.tiles > c.tiles; });
  };
  pl.items.resize(n);
  for (size_t x = 0; x < X; ++x) {
    sort_share(x * per, (x + 1) * per);
    for (size_t k = 0; k < per; ++k) pl.items[k * X + x] = v[x * per + k].it;
  }
  // The remainder (fewer than X) is dispatched last.
  sort_share(X * per, n);
  for (size_t i = X * per; i < n; ++i) pl.items[i] = v[i].it;
}

// Shapes, segment table and planning. `bwd` additionally folds aliases and
// builds the dK/dV work list. A positive `fwd_split_cap` bounds the forward's
// key-axis splits. Pure host code.
cas_status_t build_plan(const cas_problem_t *p, bool bwd, Plan &pl, int fwd_split_cap = 0) {
  if (!p) return fail(CAS_ERR_INVALID_ARGUMENT, "problem is NULL");
  // The caller may pass any integer through the C ABI: read the field's
  // bits as an integer (loading an out-of-range enumerator is undefined).
  int32_t dtype_raw = 0;
  static_assert(sizeof(p->dtype) == sizeof(dtype_raw), "cas_dtype_t is 32-bit");
  std::memcpy(&dtype_raw, &p->dtype, sizeof(dtype_raw));
  if (dtype_raw != CAS_DTYPE_BF16 && dtype_raw != CAS_DTYPE_FP32)
    return fail(CAS_ERR_INVALID_ARGUMENT, "unknown dtype");
  if (p->batch < 1 || p->num_kv_heads < 1 || p->group_size < 1 || p->head_dim < 1)
    return fail(CAS_ERR_INVALID_ARGUMENT, "batch, num_kv_heads, group_size and head_dim must be >= 1");
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(CAS_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (!std::isfinite(p->softmax_scale) || !(p->softmax_scale > 0.0f))
    return fail(CAS_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  const int64_t Hq = (int64_t)p->num_kv_heads * p->group_size;
  if (Hq > (1 << 16)) return fail(CAS_ERR_UNSUPPORTED, "num_kv_heads*group_size above 2^16");
  if ((int64_t)p->num_kv_heads * p->head_dim > (1 << 22))
    return fail(CAS_ERR_UNSUPPORTED, "num_kv_heads*head_dim above 2^22 (self-token stride)");
  // Query layout: per-row token offsets and lengths.
  pl.packed = p->q_offsets != nullptr;
  pl.tok0.resize(p->batch);
  pl.len.resize(p->batch);
  if (pl.packed) {
    if (p->q_len != 0) return fail(CAS_ERR_INVALID_ARGUMENT, "q_len must be 0 when q_offsets is given");
    if (p->q_offsets[0] != 0) return fail(CAS_ERR_INVALID_ARGUMENT, "q_offsets[0] must be 0");
    for (int b = 0; b < p->batch; ++b) {
      if (p->q_offsets[b + 1] < p->q_offsets[b])
        return fail(CAS_ERR_INVALID_ARGUMENT, "q_offsets must be non-decreasing");
      pl.tok0[b] = p->q_offsets[b];
      pl.len[b] = p->q_offsets[b + 1] - p->q_offsets[b];
    }
    pl.T = p->q_offsets[p->batch];
    if (pl.T < 1) return fail(CAS_ERR_INVALID_ARGUMENT, "packed rows hold no query token");
  } else {
    if (p->q_len < 1) return fail(CAS_ERR_INVALID_ARGUMENT, "q_len must be >= 1");
    if ((int64_t)p->batch * p->q_len > INT32_MAX)
      return fail(CAS_ERR_UNSUPPORTED, "batch*q_len above 2^31");
    for (int b = 0; b < p->batch; ++b) {
      pl.tok0[b] = b * p->q_len;
      pl.len[b] = p->q_len;
    }
    pl.T = (int64_t)p->batch * p->q_len;
    pl.Sq = p->q_len;
  }
  pl.Smax = *std::max_element(pl.len.begin(), pl.len.end());
  if (pl.T * Hq > INT32_MAX) return fail(CAS_ERR_UNSUPPORTED, "tokens*num_kv_heads*group_size above 2^31");
  if ((int64_t)p->group_size * pl.Smax > (1 << 28))
    return fail(CAS_ERR_UNSUPPORTED, "group_size*(longest row) above 2^28");
  if (pl.T * Hq * p->head_dim > (int64_t)1 << 40)
    return fail(CAS_ERR_UNSUPPORTED, "query tensor too large");
  if (!p->seg_offsets) return fail(CAS_ERR_INVALID_ARGUMENT, "seg_offsets is NULL");
  if (p->seg_offsets[0] != 0) return fail(CAS_ERR_INVALID_ARGUMENT, "seg_offsets[0] must be 0");
  for (int b = 0; b < p->batch; ++b)
    if (p->seg_offsets[b + 1] < p->seg_offsets[b])
      return fail(CAS_ERR_INVALID_ARGUMENT, "seg_offsets must be non-decreasing");
  const int32_t nent = p->seg_offsets[p->batch];
  if (nent > (1 << 20)) return fail(CAS_ERR_UNSUPPORTED, "more than 2^20 segment entries");
  if (nent > 0 && !p->segments) return fail(CAS_ERR_INVALID_ARGUMENT, "segments is NULL");

  pl.dt = dtype_raw == CAS_DTYPE_BF16 ? kBF16 : kFP32;
  pl.esize = dtype_raw == CAS_DTYPE_BF16 ? 2 : 4;
  pl.B = p->batch;
  pl.Hkv = p->num_kv_heads;
  pl.g = p->group_size;
  pl.Hq = (int)Hq;
  pl.D = p->head_dim;
  pl.nrows_max = pl.Smax * pl.g;
  pl.nqb_max = (int)ceil_div(pl.nrows_max, 64);
  pl.scale = p->softmax_scale;

  const int D = pl.D, es = pl.esize, Hkv = pl.Hkv;
  int64_t min_row_tiles = INT64_MAX;
  int64_t tblk = 0;
  pl.rows.resize(pl.B);
  for (int b = 0; b < pl.B; ++b) {
    DevRow r{};
    r.seg_begin = (int32_t)pl.segs.size();
    r.tile_begin = (int32_t)pl.tiles.size();
    r.tok0 = pl.tok0[b];
    r.len = pl.len[b];
    r.lse0 = pl.packed ? pl.tok0[b] : (int32_t)((int64_t)b * Hq * pl.Sq);
    r.tblk0 = (int32_t)tblk;
    tblk += (int64_t)Hkv * ceil_div((int64_t)pl.len[b] * pl.g, 64);
    int64_t tiles = 0, plen = 0;
    for (int i = p->seg_offsets[b]; i < p->seg_offsets[b + 1]; ++i) {
      const cas_segment_t &s = p->segments[i];
      if (s.len < 0) return fail(CAS_ERR_INVALID_ARGUMENT, "segment " + std::to_string(i) + ": negative len");
      if (s.len == 0) continue;
      if (!s.k || !s.v) return fail(CAS_ERR_INVALID_ARGUMENT, "segment " + std::to_string(i) + ": NULL k or v");
      if (s.stride_tok < 1 || s.stride_head < 0 || (Hkv > 1 && s.stride_head < 1))
        return fail(CAS_ERR_INVALID_ARGUMENT, "segment " + std::to_string(i) + ": bad strides");
      if (!aligned16(s.k) || !aligned16(s.v) || !aligned16(s.dk) || !aligned16(s.dv) ||
          (s.stride_tok * es) % 16 != 0 || (s.stride_head * es) % 16 != 0)
        return fail(CAS_ERR_ALIGNMENT, "segment " + std::to_string(i) +
                                           ": pointers and strides must be multiples of 16 bytes");
      if (s.len > (1 << 30)) return fail(CAS_ERR_UNSUPPORTED, "segment longer than 2^30 tokens");
      // Tile copies address up to 128 tokens with 32-bit byte offsets.
      if (s.stride_tok > (1 << 22))
        return fail(CAS_ERR_UNSUPPORTED, "segment " + std::to_string(i) + ": token stride above 2^22 elements");
      DevSeg d{};
      d.k = s.k;
      d.v = s.v;
      d.stride_tok = s.stride_tok;
      d.stride_head = s.stride_head;
      d.len = (int32_t)s.len;
      d.tile_begin = (int32_t)tiles;
      for (int64_t key0 = 0; key0 < s.len; key0 += kKeyTile) {
        DevTile t{};
        t.k = (const char *)s.k + key0 * s.stride_tok * es;
        t.v = (const char *)s.v + key0 * s.stride_tok * es;
        t.stride_head = s.stride_head;
        t.stride_tok = (int32_t)s.stride_tok;
        t.nvalid = (int32_t)std::min<int64_t>(kKeyTile, s.len - key0);
        pl.tiles.push_back(t);
      }
      tiles += ceil_div(s.len, kKeyTile);
      plen += s.len;
      pl.segs.push_back(d);
    }
    if (plen + pl.len[b] > (int64_t)1 << 30)
      return fail(CAS_ERR_UNSUPPORTED, "row " + std::to_string(b) + ": prefix longer than 2^30 tokens");
    r.seg_end = (int32_t)pl.segs.size();
    r.prefix_tiles = (int32_t)tiles;
    // The row's causal self tiles follow its prefix tiles; k/v hold byte
    // offsets from k_self/v_self until bind_self_tiles adds the base.
    for (int64_t s0 = 0; s0 < pl.len[b]; s0 += kKeyTile) {
      DevTile t{};
      const int64_t off = (((int64_t)pl.tok0[b] + s0) * Hkv) * D * es;
      t.k = (const void *)(uintptr_t)off;
      t.v = (const void *)(uintptr_t)off;
      t.stride_head = D;
      t.stride_tok = Hkv * D;
      t.nvalid = (int32_t)std::min<int64_t>(kKeyTile, pl.len[b] - s0);
      pl.tiles.push_back(t);
    }
    pl.rows[b] = r;
    pl.max_prefix = std::max(pl.max_prefix, plen);
    min_row_tiles = std::min(min_row_tiles, tiles + 1);
  }

  const cas_tuning_t tu = tuning();
  const bool bf16 = pl.dt == kBF16;
  const int rpw_fwd = bf16 ? kBf16RowsPerWg : kRowsPerWg, rpw_dq = bf16 ? kBf16RowsPerWg : kDqRowsPerWg;
  pl.nqblk_fwd = (int)ceil_div(pl.nrows_max, rpw_fwd);
  pl.nqblk_dq = (int)ceil_div(pl.nrows_max, rpw_dq);
  // The grids are sized for the longest row; the split heuristic counts the
  // workgroups that have rows.
  int64_t base_fwd = 0, base_dq = 0;
  for (int b = 0; b < pl.B; ++b) {
    base_fwd += Hkv * ceil_div((int64_t)pl.len[b] * pl.g, rpw_fwd);
    base_dq += Hkv * ceil_div((int64_t)pl.len[b] * pl.g, rpw_dq);
  }
  const Topology topo = device_topology();
  pl.xcds = topo.xcds;
  pl.cus = topo.cus;
  pl.fwd_splits = tu.fwd_splits > 0 ? std::min(tu.fwd_splits, kMaxSplits)
                                    : auto_splits(base_fwd, min_row_tiles, topo.cus);
  if (fwd_split_cap > 0) pl.fwd_splits = std::min(pl.fwd_splits, fwd_split_cap);
  pl.dq_splits = tu.dq_splits > 0 ? std::min(tu.dq_splits, kMaxSplits) : auto_splits(base_dq, min_row_tiles, topo.cus);
  if ((int64_t)pl.B * Hkv * pl.nqblk_fwd * pl.fwd_splits > INT32_MAX ||
      (int64_t)pl.B * Hkv * pl.nqblk_dq * pl.dq_splits > INT32_MAX)
    return fail(CAS_ERR_UNSUPPORTED, "grid too large");
  if (bf16) build_items(pl, bwd ? pl.dq_splits : pl.fwd_splits);

  if (bwd) {
    // Fold entries that name the same cartridge storage into one cartridge.
    std::map<std::tuple<uintptr_t, uintptr_t, int64_t, int64_t, int64_t>, int> index;
    std::vector<std::vector<int32_t>> users;
    std::vector<const cas_segment_t *> first;
    for (int b = 0; b < pl.B; ++b) {
      for (int i = p->seg_offsets[b]; i < p->seg_offsets[b + 1]; ++i) {
        const cas_segment_t &s = p->segments[i];
        if (s.len == 0) continue;
        auto key = std::make_tuple((uintptr_t)s.k, (uintptr_t)s.v, s.len, s.stride_tok, s.stride_head);
        auto it = index.find(key);
        int u;
        if (it == index.end()) {
          u = (int)first.size();
          index.emplace(key, u);
          first.push_back(&s);
          users.emplace_back();
        } else {
          u = it->second;
          if (first[u]->dk != s.dk || first[u]->dv != s.dv)
            return fail(CAS_ERR_INVALID_ARGUMENT, "segment " + std::to_string(i) +
                                                      ": entries sharing k/v storage must share dk/dv");
        }
        users[u].push_back(b);
      }
    }
    int64_t tiles = 0;
    for (size_t u = 0; u < first.size(); ++u) {
      const cas_segment_t &s = *first[u];
      if (!s.dk && !s.dv) continue;
      DevCart c{};
      c.k = s.k;
      c.v = s.v;
      c.dk = s.dk;
      c.dv = s.dv;
      c.stride_tok = s.stride_tok;
      c.stride_head = s.stride_head;
      c.len = (int32_t)s.len;
      c.tile_begin = (int32_t)tiles;
      c.use_begin = (int32_t)pl.uses.size();
      // Rows without queries add nothing and are left out.
      int64_t nblk = 0;
      for (int32_t b : users[u]) {
        if (pl.len[b] == 0) continue;
        pl.uses.push_back(b);
        nblk += ceil_div((int64_t)pl.len[b] * pl.g, kDkdvQBlock);
      }
      c.use_end = (int32_t)pl.uses.size();
      if (nblk > INT32_MAX) return fail(CAS_ERR_UNSUPPORTED, "too many query blocks per cartridge");
      c.nblk = (int32_t)nblk;
      tiles += ceil_div(s.len, kDkdvKeyTile);
      pl.carts.push_back(c);
      // A gradient buffer must not overlap itself under its strides.
      int64_t s1 = s.stride_tok, n1 = s.len, s2 = s.stride_head, n2 = Hkv;
      if (s1 > s2 || n1 == 1) {
        std::swap(s1, s2);
        std::swap(n1, n2);
      }
      bool ok = true;
      if (n1 > 1 && s1 < D) ok = false;
      if (n2 > 1 && (s2 < D || (n1 > 1 && s2 < s1 * n1))) ok = false;
      if (!ok)
        return fail(CAS_ERR_INVALID_ARGUMENT, "cartridge gradient layout overlaps itself");
    }
    if (tiles > INT32_MAX / 2) return fail(CAS_ERR_UNSUPPORTED, "too many key tiles");
    pl.cart_tiles = (int)tiles;
    pl.self_tiles_max = (int)ceil_div(pl.Smax, kDkdvKeyTile);
    int64_t self_tiles = 0;
    for (int b = 0; b < pl.B; ++b) self_tiles += ceil_div(pl.len[b], kDkdvKeyTile);
    pl.order_cap = (tiles + self_tiles) * Hkv;
    if (tiles + (int64_t)pl.B * pl.self_tiles_max > INT32_MAX / 2 || pl.order_cap > INT32_MAX)
      return fail(CAS_ERR_UNSUPPORTED, "too many key tiles");
  }

  // Workspace layout.
  size_t off = 0;
  pl.off_segs = off;
  off = align_up(off + pl.segs.size() * sizeof(DevSeg), 256);
  pl.off_rows = off;
  off = align_up(off + pl.rows.size() * sizeof(DevRow), 256);
  pl.off_tiles = off;
  off = align_up(off + pl.tiles.size() * sizeof(DevTile), 256);
  pl.off_items = off;
  off = align_up(off + pl.items.size() * sizeof(DevItem), 256);
  if (bwd) {
    pl.off_carts = off;
    off = align_up(off + pl.carts.size() * sizeof(DevCart), 256);
    pl.off_uses = off;
    off = align_up(off + pl.uses.size() * sizeof(int32_t), 256);
    pl.off_order = off;
    off = align_up(off + (size_t)pl.order_cap * sizeof(DevWg), 256);
    pl.off_queues = off;
    off = align_up(off + (size_t)pl.xcds * sizeof(DevQueue), 256);
    pl.off_claim = off;   // claim counters: zero in every table upload
    off = align_up(off + (size_t)pl.xcds * sizeof(int32_t), 256);
  }
  pl.table_bytes = off;
  const size_t plane = (size_t)pl.T * pl.Hq;   // packed rows of all batch rows and KV heads
  if (!bwd) {
    if (pl.fwd_splits > 1) {
      pl.off_part_o = off;
      off = align_up(off + (size_t)pl.fwd_splits * plane * D * 4, 256);
      pl.off_part_lse = off;
      off = align_up(off + (size_t)pl.fwd_splits * plane * 4, 256);
    }
    if (pl.dt == kBF16) {
      // Per-workgroup flags of the exact (online-softmax) pass.
      pl.off_ovf = off;
      off = align_up(off + (size_t)pl.B * Hkv * pl.nqblk_fwd * pl.fwd_splits * 4, 256);
    }
    pl.ws_fwd = off;
  } else {
    pl.off_nd = off;
    off = align_up(off + plane * 4, 256);
    pl.off_lse2 = off;
    off = align_up(off + plane * 4, 256);
    if (pl.dt == kBF16) {
      // Transposed Q and dO of every 64-row block (dK/dV operands).
      const size_t tbytes = (size_t)tblk * 64 * D * 2;
      pl.off_qT = off;
      off = align_up(off + tbytes, 256);
      pl.off_doT = off;
      off = align_up(off + tbytes, 256);
    }
    if (pl.dq_splits > 1) {
      pl.off_part_dq = off;
      off = align_up(off + (size_t)pl.dq_splits * plane * D * 4, 256);
    }
    pl.ws_bwd = off;
  }
  return CAS_OK;
}

// dK/dV workgroup list: every cartridge tile (and, with self gradients, every
// self tile of every row) at every KV head, sorted by the number of 64-row
// query blocks the workgroup walks, most first; ties go by KV head, then by
// the tile's position within its cartridge (or the row's self keys), then
// tile order. Longest-first dispatch keeps the long workgroups off the tail;
// the position tie-break lets the workgroups that run side by side on an XCD
// come from all the cartridges (and so rows) of their KV head, instead of
// all walking one row's query blocks.
void build_dkdv_order(Plan &pl, bool with_self) {
  struct E {
    int64_t nblk;
    int32_t tile, kvh, pos;   // pos: tile within its cartridge or the row's self keys
  };
  std::vector<E> v;
  v.reserve((size_t)pl.order_cap);
  for (const DevCart &c : pl.carts) {
    const int n = (int)ceil_div(c.len, kDkdvKeyTile);
    for (int kvh = 0; kvh < pl.Hkv; ++kvh)
      for (int t = 0; t < n; ++t) v.push_back({c.nblk, c.tile_begin + t, kvh, t});
  }
  if (with_self) {
    for (int b = 0; b < pl.B; ++b) {
      const int64_t nqb = ceil_div((int64_t)pl.len[b] * pl.g, kDkdvQBlock);
      const int n = (int)ceil_div(pl.len[b], kDkdvKeyTile);
      for (int kvh = 0; kvh < pl.Hkv; ++kvh)
        for (int j = 0; j < n; ++j)
          v.push_back({nqb - ((int64_t)j * kDkdvKeyTile * pl.g) / kDkdvQBlock,
                       pl.cart_tiles + b * pl.self_tiles_max + j, kvh, j});
    }
  }
  std::stable_sort(v.begin(), v.end(), [](const E &a, const E &b) {
    if (a.nblk != b.nblk) return a.nblk > b.nblk;
    if (a.kvh != b.kvh) return a.kvh < b.kvh;
    if (a.pos != b.pos) return a.pos < b.pos;
    return a.tile < b.tile;
  });
  pl.order.resize(v.size());
  pl.queues.clear();
  pl.dkdv_grid = (int64_t)v.size();
  const int X = pl.xcds;
  if (v.empty()) return;
  if (X > 1 && pl.Hkv % X == 0) {
    // XCD-affine: workgroup i runs on XCD i % X (round-robin dispatch), and
    // XCD x takes the entries of KV heads h with h % X == x, longest first.
    // Every KV head has the same tiles, so the X lists are equally long; the
    // query blocks of one (row, KV head) are then streamed by one XCD's L2.
    std::vector<std::vector<E>> q(X);
    for (const E &e : v) q[e.kvh % X].push_back(e);
    const int64_t per_cu = std::max(1, pl.cus / X);   // CUs of one XCD
    const int64_t cnt = (int64_t)q[0].size();
    if (pl.dt == kBF16 && (int64_t)X * (cnt + per_cu) <= INT32_MAX) {
      // Each XCD's list in one piece: a static head, taken by workgroup
      // index, and a tail of its shortest entries (two rounds of the XCD's
      // CUs, or an eighth of the list) claimed at run time, by the XCD's own
      // workgroups first and then by XCDs that finished their own lists; one
      // more round of workgroups per XCD is launched for that. XCDs run at
      // different speeds (up to 4 % apart on one chip), so a fixed share per
      // XCD ends with the slowest.
      const int64_t tail = std::min(cnt, std::max(2 * per_cu, cnt / 8));
      pl.queues.resize(X);
      size_t at = 0;
      for (int x = 0; x < X; ++x) {
        pl.queues[x] = {(int32_t)at, (int32_t)cnt, (int32_t)(cnt - tail), 0};
        for (const E &e : q[x]) pl.order[at++] = {e.tile, e.kvh};
      }
      pl.dkdv_grid = (int64_t)X * (cnt + per_cu);
      return;
    }
    std::vector<size_t> next(X, 0);
    for (size_t i = 0; i < v.size(); ++i) {
      const E &e = q[i % X][next[i % X]++];
      pl.order[i] = {e.tile, e.kvh};
    }
    return;
  }
  for (size_t i = 0; i < v.size(); ++i) pl.order[i] = {v[i].tile, v[i].kvh};
}

// Turns the self-tile offsets of the tile table into pointers.
void bind_self_tiles(Plan &pl, const void *k_self, const void *v_self) {
  for (int b = 0; b < pl.B; ++b) {
    const DevRow &r = pl.rows[b];
    const int n = (int)ceil_div(pl.len[b], kKeyTile);
    for (int i = 0; i < n; ++i) {
      DevTile &t = pl.tiles[r.tile_begin + r.prefix_tiles + i];
      t.k = (const char *)k_self + (uintptr_t)t.k;
      t.v = (const char *)v_self + (uintptr_t)t.v;
    }
  }
}

void add_segment_intervals(const Plan &pl, const cas_problem_t *p, bool with_grads,
                           std::vector<Interval> &iv) {
  const int es = pl.esize;
  for (int i = 0; i < p->seg_offsets[p->batch]; ++i) {
    const cas_segment_t &s = p->segments[i];
    if (s.len == 0) continue;
    const uintptr_t span = (uintptr_t)(((s.len - 1) * s.stride_tok + (pl.Hkv - 1) * s.stride_head + pl.D) * es);
    iv.push_back({(uintptr_t)s.k, (uintptr_t)s.k + span, false, 0, "segment k"});
    iv.push_back({(uintptr_t)s.v, (uintptr_t)s.v + span, false, 0, "segment v"});
    if (with_grads) {
      // Entries of one aliased cartridge carry identical (dk, dv) intervals.
      if (s.dk) iv.push_back({(uintptr_t)s.dk, (uintptr_t)s.dk + span, true, (uintptr_t)s.dk, "segment dk"});
      if (s.dv) iv.push_back({(uintptr_t)s.dv, (uintptr_t)s.dv + span, true, (uintptr_t)s.dv, "segment dv"});
    }
  }
}

// ---------------------------------------------------------------------------
// Pinned staging ring for launch tables (host -> workspace, copied by a
// small kernel on the launch stream).
// ---------------------------------------------------------------------------
constexpr size_t kMinSlotBytes = 1 << 20;
constexpr int kSlots = 8;

struct Ring {
  char *host = nullptr;
  size_t slot_bytes = 0;
  hipEvent_t ev[kSlots] = {};
  bool used[kSlots] = {};
  int next = 0;
};

std::mutex g_ring_mu;
std::map<int, Ring> g_rings;

// Copies `bytes` of launch tables, written by fill() into a pinned slot,
// to the workspace on the stream.
template <typename Fill>
cas_status_t ring_upload(size_t bytes, void *ws, hipStream_t stream, Fill &&fill) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_ring_mu);
  Ring &r = g_rings[dev];
  if (!r.ev[0]) {
    for (int i = 0; i < kSlots; ++i) {
      e = hipEventCreateWithFlags(&r.ev[i], hipEventDisableTiming);
      if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(e));
    }
  }
  if (!r.host || bytes > r.slot_bytes) {
    // (Re)allocate the pinned ring once every earlier upload from it is done.
    for (int i = 0; i < kSlots; ++i) {
      if (!r.used[i]) continue;
      e = hipEventSynchronize(r.ev[i]);
      if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("hipEventSynchronize: ") + hipGetErrorString(e));
      r.used[i] = false;
    }
    if (r.host) {
      e = hipHostFree(r.host);
      r.host = nullptr;
      r.slot_bytes = 0;
      if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("hipHostFree: ") + hipGetErrorString(e));
    }
    size_t sb = kMinSlotBytes;
    while (sb < bytes) sb *= 2;
    // Coherent: the upload kernel reads the slots the host has just
    // rewritten, so no GPU cache may keep an earlier upload's lines.
    e = hipHostMalloc((void **)&r.host, sb * kSlots, hipHostMallocCoherent);
    if (e != hipSuccess) {
      r.host = nullptr;
      r.slot_bytes = 0;
      return fail(CAS_ERR_HIP, std::string("hipHostMalloc: ") + hipGetErrorString(e));
    }
    r.slot_bytes = sb;
  }
  const int slot = r.next;
  r.next = (r.next + 1) % kSlots;
  if (r.used[slot]) {
    e = hipEventSynchronize(r.ev[slot]);
    if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("hipEventSynchronize: ") + hipGetErrorString(e));
  }
  char *h = r.host + (size_t)slot * r.slot_bytes;
  std::memset(h, 0, bytes);
  fill(h);
  e = launch_table_upload(ws, h, bytes, stream);
  if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("table upload launch: ") + hipGetErrorString(e));
  e = hipEventRecord(r.ev[slot], stream);
  if (e != hipSuccess) return fail(CAS_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
  r.used[slot] = true;
  return CAS_OK;
}

// Writes the launch tables, laid out as in the workspace, to host memory h
// (table_bytes, zeroed by the caller).
void fill_tables(const Plan &pl, bool bwd, char *h) {
  if (!pl.segs.empty()) std::memcpy(h + pl.off_segs, pl.segs.data(), pl.segs.size() * sizeof(DevSeg));
  std::memcpy(h + pl.off_rows, pl.rows.data(), pl.rows.size() * sizeof(DevRow));
  if (!pl.tiles.empty()) std::memcpy(h + pl.off_tiles, pl.tiles.data(), pl.tiles.size() * sizeof(DevTile));
  if (!pl.items.empty()) std::memcpy(h + pl.off_items, pl.items.data(), pl.items.size() * sizeof(DevItem));
  if (bwd) {
    if (!pl.carts.empty()) std::memcpy(h + pl.off_carts, pl.carts.data(), pl.carts.size() * sizeof(DevCart));
    if (!pl.uses.empty()) std::memcpy(h + pl.off_uses, pl.uses.data(), pl.uses.size() * sizeof(int32_t));
    if (!pl.order.empty()) std::memcpy(h + pl.off_order, pl.order.data(), pl.order.size() * sizeof(DevWg));
    if (!pl.queues.empty())
      std::memcpy(h + pl.off_queues, pl.queues.data(), pl.queues.size() * sizeof(DevQueue));
  }
}

cas_status_t upload_tables(const Plan &pl, bool bwd, void *ws, hipStream_t stream) {
  return ring_upload(pl.table_bytes, ws, stream, [&](char *h) { fill_tables(pl, bwd, h); });
}

// ---------------------------------------------------------------------------
// Cartridge Adam step: validation and launch tables.
// ---------------------------------------------------------------------------
struct AdamPlan {
  std::vector<DevAdamT> tensors;
  std::vector<DevAdamChunk> chunks;
  size_t off_chunks = 0, bytes = 0;
};

float lr_scale(int32_t step, int32_t warmup, int32_t buckets) {
  if (buckets < 1 || step < 0) return NAN;
  if (warmup <= 0 || step >= warmup) return 1.0f;
  // ceil(buckets * step / warmup), at least the first level
  const int64_t lvl = std::max<int64_t>(1, ((int64_t)buckets * step + warmup - 1) / warmup);
  return (float)std::min<int64_t>(lvl, buckets) / (float)buckets;
}

cas_status_t build_adam(const cas_adam_cartridge_t *carts, int32_t n, int32_t Hkv, int32_t D,
                        const cas_adam_config_t *cfg, AdamPlan &ap) {
  if (n < 0) return fail(CAS_ERR_INVALID_ARGUMENT, "n must be >= 0");
  if (n > 0 && !carts) return fail(CAS_ERR_INVALID_ARGUMENT, "carts is NULL");
  if (Hkv < 1) return fail(CAS_ERR_INVALID_ARGUMENT, "num_kv_heads must be >= 1");
  if (D != 64 && D != 128) return fail(CAS_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (cfg) {
    if (!std::isfinite(cfg->lr) || cfg->lr < 0.0f) return fail(CAS_ERR_INVALID_ARGUMENT, "lr must be finite and >= 0");
    if (!(cfg->beta1 >= 0.0f && cfg->beta1 < 1.0f) || !(cfg->beta2 >= 0.0f && cfg->beta2 < 1.0f))
      return fail(CAS_ERR_INVALID_ARGUMENT, "beta1 and beta2 must lie in [0, 1)");
    if (!std::isfinite(cfg->eps) || !(cfg->eps > 0.0f)) return fail(CAS_ERR_INVALID_ARGUMENT, "eps must be finite and > 0");
    if (cfg->warmup_buckets < 1 || cfg->warmup_steps < 0)
      return fail(CAS_ERR_INVALID_ARGUMENT, "warmup_buckets must be >= 1 and warmup_steps >= 0");
  }
  std::vector<Interval> iv;
  for (int i = 0; i < n; ++i) {
    const cas_adam_cartridge_t &c = carts[i];
    const std::string who = "cartridge " + std::to_string(i);
    if (c.len < 0 || c.step < 0 || c.frozen_tokens < 0)
      return fail(CAS_ERR_INVALID_ARGUMENT, who + ": len, step and frozen_tokens must be >= 0");
    if (c.len > (1 << 30)) return fail(CAS_ERR_UNSUPPORTED, who + ": longer than 2^30 tokens");
    if (c.len <= c.frozen_tokens) continue;   // nothing to update
    const void *ptrs[8] = {c.k, c.v, c.dk, c.dv, c.m1_k, c.m2_k, c.m1_v, c.m2_v};
    for (const void *q : ptrs)
      if (!q) return fail(CAS_ERR_INVALID_ARGUMENT, who + ": NULL tensor");
    for (const void *q : ptrs)
      if (!aligned16(q)) return fail(CAS_ERR_ALIGNMENT, who + ": tensors must be 16-byte aligned");
    if (c.stride_tok < 1 || c.stride_head < 0 || (Hkv > 1 && c.stride_head < 1))
      return fail(CAS_ERR_INVALID_ARGUMENT, who + ": bad strides");
    if (c.stride_tok % 8 != 0 || c.stride_head % 8 != 0)
      return fail(CAS_ERR_ALIGNMENT, who + ": strides must be multiples of 8 elements");
    int64_t s1 = c.stride_tok, n1 = c.len, s2 = c.stride_head, n2 = Hkv;
    if (s1 > s2 || n1 == 1) {
      std::swap(s1, s2);
      std::swap(n1, n2);
    }
    if ((n1 > 1 && s1 < D) || (n2 > 1 && (s2 < D || (n1 > 1 && s2 < s1 * n1))))
      return fail(CAS_ERR_INVALID_ARGUMENT, who + ": parameter layout overlaps itself");
    const uintptr_t span = (uintptr_t)(((c.len - 1) * c.stride_tok + (int64_t)(Hkv - 1) * c.stride_head + D) * 2);
    const uintptr_t mom = (uintptr_t)c.len * Hkv * D * 4;
    // Every written tensor is its own owner: no two may overlap, even at equal addresses.
    const uintptr_t own = (uintptr_t)i * 8 + 1;
    iv.push_back({(uintptr_t)c.k, (uintptr_t)c.k + span, true, own, "k"});
    iv.push_back({(uintptr_t)c.v, (uintptr_t)c.v + span, true, own + 1, "v"});
    iv.push_back({(uintptr_t)c.dk, (uintptr_t)c.dk + span, false, 0, "dk"});
    iv.push_back({(uintptr_t)c.dv, (uintptr_t)c.dv + span, false, 0, "dv"});
    int j = 2;
    for (float *m : {c.m1_k, c.m2_k, c.m1_v, c.m2_v})
      iv.push_back({(uintptr_t)m, (uintptr_t)m + mom, true, own + j++, "moment"});
  }
  std::string msg;
  if (!overlap_free(iv, msg)) return fail(CAS_ERR_INVALID_ARGUMENT, msg);
  for (int i = 0; i < n; ++i) {
    const cas_adam_cartridge_t &c = carts[i];
    if (c.len <= c.frozen_tokens) continue;
    const double t = (double)c.step + 1.0;
    for (int which = 0; which < 2; ++which) {
      DevAdamT d{};
      d.x = (__bf16 *)(which ? c.v : c.k);
      d.g = (const __bf16 *)(which ? c.dv : c.dk);
      d.m1 = which ? c.m1_v : c.m1_k;
      d.m2 = which ? c.m2_v : c.m2_k;
      d.stride_tok = c.stride_tok;
      d.stride_head = c.stride_head;
      d.len = (int32_t)c.len;
      d.frozen = c.frozen_tokens;
      if (cfg) {
        d.lr = cfg->lr * lr_scale(c.step, cfg->warmup_steps, cfg->warmup_buckets);
        d.bc1 = (float)(1.0 - std::pow((double)cfg->beta1, t));
        d.bc2 = (float)(1.0 - std::pow((double)cfg->beta2, t));
      }
      const int32_t ti = (int32_t)ap.tensors.size();
      ap.tensors.push_back(d);
      for (int64_t tok = c.frozen_tokens; tok < c.len; tok += kAdamChunk) ap.chunks.push_back({ti, (int32_t)tok});
    }
    if (ap.chunks.size() > (size_t)INT32_MAX) return fail(CAS_ERR_UNSUPPORTED, "too many chunks");
  }
  ap.off_chunks = align_up(ap.tensors.size() * sizeof(DevAdamT), 256);
  ap.bytes = align_up(ap.off_chunks + ap.chunks.size() * sizeof(DevAdamChunk), 256);
  return CAS_OK;
}

// ---------------------------------------------------------------------------
// Optional per-kernel timing.
// ---------------------------------------------------------------------------
struct TimedLaunch {
  const char *name;
  hipEvent_t a, b;
};

std::mutex g_time_mu;
bool g_timing = false;
std::vector<TimedLaunch> g_pending;
std::vector<hipEvent_t> g_event_pool;
std::map<std::string, std::pair<int, double>> g_totals;

hipEvent_t pooled_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
hipError_t timed(const char *name, hipStream_t s, F &&launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lk(g_time_mu);
    on = g_timing;
  }
  if (!on) return launch();
  hipEvent_t a, b;
  {
    std::lock_guard<std::mutex> lk(g_time_mu);
    a = pooled_event();
    b = pooled_event();
  }
  if (!a || !b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, s);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, s);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_time_mu);
  g_pending.push_back({name, a, b});
  return hipSuccess;
}

cas_status_t hip_fail(const char *what, hipError_t e) {
  return fail(CAS_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

cas_status_t check_workspace(void *ws, size_t have, size_t need) {
  if (need > 0 && !ws) return fail(CAS_ERR_WORKSPACE, "workspace is NULL");
  if (have < need)
    return fail(CAS_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes, have " +
                                       std::to_string(have));
  if (!aligned16(ws)) return fail(CAS_ERR_ALIGNMENT, "workspace must be 16-byte aligned");
  return CAS_OK;
}

// ---------------------------------------------------------------------------
// Paged decode: validation, key-axis split planning and launch tables.
// ---------------------------------------------------------------------------
constexpr int kMaxDecSplits = 64;

struct DecodePlan {
  int Tq = 0, Hq = 0;
  std::vector<DevDecodeReq> reqs;
  std::vector<DevDecodeWork> work;
  std::vector<int32_t> tok_req;
  int max_split = 1;
  size_t off_work = 0, off_pages = 0, off_tokreq = 0, off_plse = 0, off_po = 0, bytes = 0;
};

cas_status_t build_decode(const cas_decode_problem_t *p, DecodePlan &dp) {
  if (!p) return fail(CAS_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (p->batch < 1 || p->num_kv_heads < 1 || p->group_size < 1)
    return fail(CAS_ERR_INVALID_ARGUMENT, "batch, num_kv_heads and group_size must be >= 1");
  if (p->head_dim != 64 && p->head_dim != 128) return fail(CAS_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (!std::isfinite(p->softmax_scale) || !(p->softmax_scale > 0.0f))
    return fail(CAS_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  const int P = p->page_size;
  if (P != 16 && P != 32 && P != 64 && P != 128) return fail(CAS_ERR_UNSUPPORTED, "page_size must be 16, 32, 64 or 128");
  const int64_t Hq = (int64_t)p->num_kv_heads * p->group_size;
  if (Hq > (1 << 16)) return fail(CAS_ERR_UNSUPPORTED, "num_kv_heads*group_size above 2^16");
  if ((int64_t)P * p->num_kv_heads * p->head_dim * 2 >= ((int64_t)1 << 31))
    return fail(CAS_ERR_UNSUPPORTED, "page larger than 2 GiB");
  if (p->num_pages < 1) return fail(CAS_ERR_INVALID_ARGUMENT, "num_pages must be >= 1");
  if (!p->q_offsets || !p->kv_lens || !p->page_offsets || !p->page_ids)
    return fail(CAS_ERR_INVALID_ARGUMENT, "q_offsets, kv_lens, page_offsets and page_ids must be non-NULL");
  if (p->q_offsets[0] != 0 || p->page_offsets[0] != 0)
    return fail(CAS_ERR_INVALID_ARGUMENT, "q_offsets[0] and page_offsets[0] must be 0");
  const int B = p->batch;
  for (int b = 0; b < B; ++b) {
    const int64_t n = (int64_t)p->q_offsets[b + 1] - p->q_offsets[b];
    const int64_t L = p->kv_lens[b];
    if (n < 1) return fail(CAS_ERR_INVALID_ARGUMENT, "request " + std::to_string(b) + ": no query token");
    if (L < n) return fail(CAS_ERR_INVALID_ARGUMENT, "request " + std::to_string(b) + ": kv_len below its query count");
    if (L > (1 << 30)) return fail(CAS_ERR_UNSUPPORTED, "request " + std::to_string(b) + ": more than 2^30 keys");
    if ((int64_t)p->page_offsets[b + 1] - p->page_offsets[b] != ceil_div(L, P))
      return fail(CAS_ERR_INVALID_ARGUMENT, "request " + std::to_string(b) + ": page count must be ceil(kv_len / page_size)");
  }
  const int64_t Tq = p->q_offsets[B];
  if (Tq * Hq > INT32_MAX) return fail(CAS_ERR_UNSUPPORTED, "query tokens * heads above 2^31");
  for (int32_t i = 0; i < p->page_offsets[B]; ++i)
    if (p->page_ids[i] < 0 || p->page_ids[i] >= p->num_pages)
      return fail(CAS_ERR_INVALID_ARGUMENT, "page id " + std::to_string(i) + " out of range");
  dp.Tq = (int)Tq;
  dp.Hq = (int)Hq;
  const int g = p->group_size, Hkv = p->num_kv_heads;
  // Split planning: workgroups of at least 8 tiles (two per wave), about as
  // many as the compute units hold at once (two each), so the whole step
  // runs in one round of workgroups when the requests allow it.
  int64_t total = 0;
  for (int b = 0; b < B; ++b) {
    const int64_t n = p->q_offsets[b + 1] - p->q_offsets[b];
    total += ceil_div(p->kv_lens[b], kDecTile) * Hkv * ceil_div(n * g, kDecRows);
  }
  const int64_t per_wg = std::max<int64_t>(8, ceil_div(total, 2 * (int64_t)device_topology().cus));
  dp.reqs.resize(B);
  dp.tok_req.resize(Tq);
  struct W {
    int64_t tiles;
    DevDecodeWork w;
  };
  std::vector<W> work;
  for (int b = 0; b < B; ++b) {
    const int n = p->q_offsets[b + 1] - p->q_offsets[b];
    const int64_t nt = ceil_div(p->kv_lens[b], kDecTile);
    const int ns = (int)std::min<int64_t>(kMaxDecSplits, ceil_div(nt, per_wg));
    DevDecodeReq &r = dp.reqs[b];
    r.q0 = p->q_offsets[b];
    r.n = n;
    r.kv_len = p->kv_lens[b];
    r.page0 = p->page_offsets[b];
    r.nsplit = ns;
    dp.max_split = std::max(dp.max_split, ns);
    for (int t = 0; t < n; ++t) dp.tok_req[r.q0 + t] = b;
    for (int kvh = 0; kvh < Hkv; ++kvh)
      for (int row0 = 0; row0 < n * g; row0 += kDecRows)
        for (int s = 0; s < ns; ++s) {
          DevDecodeWork d{};
          d.b = b;
          d.kvh = kvh;
          d.row0 = row0;
          d.split = ns > 1 ? s : -1;
          d.tile0 = (int)(nt * s / ns);
          d.tile1 = (int)(nt * (s + 1) / ns);
          work.push_back({d.tile1 - d.tile0, d});
        }
  }
  if (work.size() > (size_t)INT32_MAX) return fail(CAS_ERR_UNSUPPORTED, "too many workgroups");
  // Longest ranges first.
  std::stable_sort(work.begin(), work.end(), [](const W &a, const W &b) { return a.tiles > b.tiles; });
  dp.work.resize(work.size());
  for (size_t i = 0; i < work.size(); ++i) dp.work[i] = work[i].w;
  size_t off = align_up(dp.reqs.size() * sizeof(DevDecodeReq), 256);
  dp.off_work = off;
  off = align_up(off + dp.work.size() * sizeof(DevDecodeWork), 256);
  dp.off_pages = off;
  off = align_up(off + (size_t)p->page_offsets[B] * sizeof(int32_t), 256);
  dp.off_tokreq = off;
  off = align_up(off + (size_t)Tq * sizeof(int32_t), 256);
  const size_t table_end = off;
  if (dp.max_split > 1) {
    const size_t plane = (size_t)Tq * Hq;
    dp.off_plse = off;
    off = align_up(off + (size_t)dp.max_split * plane * 4, 256);
    dp.off_po = off;
    off = align_up(off + (size_t)dp.max_split * plane * p->head_dim * 4, 256);
  }
  dp.bytes = off;
  (void)table_end;
  return CAS_OK;
}

}  // namespace

namespace cas {

cas_status_t set_error(cas_status_t s, const std::string &msg) { return fail(s, msg); }

cas_status_t set_hip_error(const char *what, hipError_t e) { return hip_fail(what, e); }

hipError_t enqueue_copies(const HostCopy *c, int n, hipMemcpyKind kind, hipStream_t s) {
  const char *run_src = nullptr;
  char *run_dst = nullptr;
  size_t run_bytes = 0;
  auto flush = [&]() -> hipError_t {
    hipError_t e = hipSuccess;
    if (run_bytes) e = hipMemcpyAsync(run_dst, run_src, run_bytes, kind, s);
    run_bytes = 0;
    return e;
  };
  for (int i = 0; i < n; ++i) {
    if (c[i].bytes == 0) continue;
    const char *src = (const char *)c[i].src;
    char *dst = (char *)c[i].dst;
    if (run_bytes && src == run_src + run_bytes && dst == run_dst + run_bytes) {
      run_bytes += c[i].bytes;
      continue;
    }
    hipError_t e = flush();
    if (e != hipSuccess) return e;
    run_src = src;
    run_dst = dst;
    run_bytes = c[i].bytes;
  }
  return flush();
}

cas_status_t prefix_attn_fwd_run(const cas_problem_t *p, const void *q, const void *k_self,
                                 const void *v_self, void *o, float *lse, void *workspace,
                                 size_t ws_bytes, hipStream_t stream, ScratchAddressFn scratch) {
  Plan pl;
  cas_status_t s = build_plan(p, false, pl);
  if (s != CAS_OK) return s;
  if (scratch) {
    // The workspace is the fixed scratch: fewer key-axis splits (smaller
    // partials) until it fits. Only the rounding order of the merge changes.
    while (pl.ws_fwd > ws_bytes && pl.fwd_splits > 1) {
      // Bytes per split (partials and flags) from this plan; the rebuilt
      // plan is checked again since each region is rounded up to 256 bytes.
      const size_t per_split = (pl.ws_fwd - pl.table_bytes) / (size_t)pl.fwd_splits;
      const size_t room = ws_bytes > pl.table_bytes ? ws_bytes - pl.table_bytes : 0;
      size_t cap = per_split ? room / per_split : 1;
      cap = std::max<size_t>(1, std::min<size_t>(cap, (size_t)pl.fwd_splits - 1));
      pl = Plan{};
      s = build_plan(p, false, pl, (int)cap);
      if (s != CAS_OK) return s;
    }
    if (pl.ws_fwd > ws_bytes)
      return fail(CAS_ERR_UNSUPPORTED, "launch tables need " + std::to_string(pl.ws_fwd) +
                                           " bytes, above the " + std::to_string(ws_bytes) +
                                           "-byte scratch of the no-allocation forward");
  }
  if (!q || !k_self || !v_self || !o) return fail(CAS_ERR_INVALID_ARGUMENT, "q, k_self, v_self and o must be non-NULL");
  if (!aligned16(q) || !aligned16(k_self) || !aligned16(v_self) || !aligned16(o) || ((uintptr_t)lse & 3u))
    return fail(CAS_ERR_ALIGNMENT, "tensors must be 16-byte aligned (lse 4-byte)");
  const uintptr_t qbytes = (uintptr_t)pl.T * pl.Hq * pl.D * pl.esize;
  const uintptr_t kvbytes = (uintptr_t)pl.T * pl.Hkv * pl.D * pl.esize;
  std::vector<Interval> iv;
  iv.push_back({(uintptr_t)q, (uintptr_t)q + qbytes, false, 0, "q"});
  iv.push_back({(uintptr_t)k_self, (uintptr_t)k_self + kvbytes, false, 0, "k_self"});
  iv.push_back({(uintptr_t)v_self, (uintptr_t)v_self + kvbytes, false, 0, "v_self"});
  iv.push_back({(uintptr_t)o, (uintptr_t)o + qbytes, true, (uintptr_t)o, "o"});
  if (lse) iv.push_back({(uintptr_t)lse, (uintptr_t)lse + (uintptr_t)pl.T * pl.Hq * 4, true, (uintptr_t)lse, "lse"});
  add_segment_intervals(pl, p, false, iv);
  std::string msg;
  if (!overlap_free(iv, msg)) return fail(CAS_ERR_INVALID_ARGUMENT, msg);
  if (scratch) {
    // Everything is validated: only now touch the device.
    hipError_t e = scratch(&workspace);
    if (e != hipSuccess) return hip_fail("hipGetSymbolAddress (no-allocation scratch)", e);
  } else {
    s = check_workspace(workspace, ws_bytes, pl.ws_fwd);
    if (s != CAS_OK) return s;
  }

  bind_self_tiles(pl, k_self, v_self);
  if (scratch) {
    // No pinned staging ring: the tables travel as kernel arguments.
    std::vector<char> h(pl.table_bytes, 0);
    fill_tables(pl, false, h.data());
    hipError_t e = launch_table_args_upload(h.data(), pl.table_bytes, workspace, stream);
    if (e != hipSuccess) return hip_fail("table upload launch", e);
  } else {
    s = upload_tables(pl, false, workspace, stream);
    if (s != CAS_OK) return s;
  }
  // Kernel timing records pooled events, which the no-allocation path must
  // not create: it launches directly.
  auto launch = [&](const char *name, auto &&f) -> hipError_t {
    return scratch ? f() : timed(name, stream, f);
  };
  char *ws = (char *)workspace;
  FwdParams fp{};
  fp.q = q;
  fp.k_self = k_self;
  fp.v_self = v_self;
  fp.o = o;
  fp.lse = lse;
  fp.part_o = pl.fwd_splits > 1 ? (float *)(ws + pl.off_part_o) : nullptr;
  fp.part_lse = pl.fwd_splits > 1 ? (float *)(ws + pl.off_part_lse) : nullptr;
  fp.segs = (const DevSeg *)(ws + pl.off_segs);
  fp.rows = (const DevRow *)(ws + pl.off_rows);
  fp.tiles = (const DevTile *)(ws + pl.off_tiles);
  fp.items = (const DevItem *)(ws + pl.off_items);
  fp.ovf_flag = pl.dt == kBF16 ? (int32_t *)(ws + pl.off_ovf) : nullptr;
  fp.plane = pl.T * pl.Hq;
  fp.B = pl.B;
  fp.Smax = pl.Smax;
  fp.Hkv = pl.Hkv;
  fp.g = pl.g;
  fp.nrows_max = pl.nrows_max;
  fp.nqblk = pl.nqblk_fwd;
  fp.splits = pl.fwd_splits;
  fp.lse_hs = pl.packed ? (int32_t)pl.T : pl.Sq;
  fp.n_items = (int32_t)pl.items.size();
  fp.scale_log2 = pl.scale * 1.4426950408889634f;
  hipError_t e = launch("fwd", [&] { return launch_fwd(fp, pl.dt, pl.D, stream); });
  if (e != hipSuccess) return hip_fail("fwd launch", e);
  if (pl.fwd_splits > 1) {
    MergeParams mp{};
    mp.part_o = fp.part_o;
    mp.part_lse = fp.part_lse;
    mp.o = o;
    mp.lse = lse;
    mp.rows = fp.rows;
    mp.plane = fp.plane;
    mp.B = pl.B;
    mp.Hkv = pl.Hkv;
    mp.g = pl.g;
    mp.nrows_max = pl.nrows_max;
    mp.splits = pl.fwd_splits;
    mp.lse_hs = fp.lse_hs;
    e = launch("fwd_merge", [&] { return launch_fwd_merge(mp, pl.dt, pl.D, stream); });
    if (e != hipSuccess) return hip_fail("fwd_merge launch", e);
  }
  return CAS_OK;
}

}  // namespace cas

extern "C" {

int32_t cas_abi_version(void) { return CAS_ABI_VERSION; }

const char *cas_status_string(cas_status_t s) {
  switch (s) {
    case CAS_OK: return "CAS_OK";
    case CAS_ERR_INVALID_ARGUMENT: return "CAS_ERR_INVALID_ARGUMENT";
    case CAS_ERR_UNSUPPORTED: return "CAS_ERR_UNSUPPORTED";
    case CAS_ERR_ALIGNMENT: return "CAS_ERR_ALIGNMENT";
    case CAS_ERR_NOT_PINNED: return "CAS_ERR_NOT_PINNED";
    case CAS_ERR_WORKSPACE: return "CAS_ERR_WORKSPACE";
    case CAS_ERR_HIP: return "CAS_ERR_HIP";
    case CAS_ERR_IO: return "CAS_ERR_IO";
  }
  return "CAS_ERR_UNKNOWN";
}

const char *cas_last_error_message(void) { return g_err.c_str(); }

float cas_adam_lr_scale(int32_t step, int32_t warmup_steps, int32_t warmup_buckets) {
  return lr_scale(step, warmup_steps, warmup_buckets);
}

cas_status_t cas_paged_decode_workspace_size(const cas_decode_problem_t *p, size_t *bytes) {
  if (!bytes) return fail(CAS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  DecodePlan dp;
  cas_status_t s = build_decode(p, dp);
  if (s != CAS_OK) return s;
  *bytes = dp.bytes;
  return CAS_OK;
}

cas_status_t cas_paged_decode_fwd(const cas_decode_problem_t *p, const void *q, const void *k_pages,
                                  const void *v_pages, void *o, float *lse, void *workspace,
                                  size_t ws_bytes, void *hip_stream) {
  DecodePlan dp;
  cas_status_t s = build_decode(p, dp);
  if (s != CAS_OK) return s;
  if (!q || !k_pages || !v_pages || !o) return fail(CAS_ERR_INVALID_ARGUMENT, "q, k_pages, v_pages and o must be non-NULL");
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(o) || ((uintptr_t)lse & 3u))
    return fail(CAS_ERR_ALIGNMENT, "tensors must be 16-byte aligned (lse 4-byte)");
  const uintptr_t qbytes = (uintptr_t)dp.Tq * dp.Hq * p->head_dim * 2;
  const uintptr_t pool = (uintptr_t)p->num_pages * p->page_size * p->num_kv_heads * p->head_dim * 2;
  std::vector<Interval> iv;
  iv.push_back({(uintptr_t)q, (uintptr_t)q + qbytes, false, 0, "q"});
  iv.push_back({(uintptr_t)k_pages, (uintptr_t)k_pages + pool, false, 0, "k_pages"});
  iv.push_back({(uintptr_t)v_pages, (uintptr_t)v_pages + pool, false, 0, "v_pages"});
  iv.push_back({(uintptr_t)o, (uintptr_t)o + qbytes, true, 1, "o"});
  if (lse) iv.push_back({(uintptr_t)lse, (uintptr_t)lse + (uintptr_t)dp.Tq * dp.Hq * 4, true, 2, "lse"});
  std::string msg;
  if (!overlap_free(iv, msg)) return fail(CAS_ERR_INVALID_ARGUMENT, msg);
  s = check_workspace(workspace, ws_bytes, dp.bytes);
  if (s != CAS_OK) return s;
  hipStream_t stream = (hipStream_t)hip_stream;
  char *ws = (char *)workspace;
  const int npage_ids = p->page_offsets[p->batch];
  s = ring_upload(dp.off_plse ? dp.off_plse : dp.bytes, workspace, stream, [&](char *h) {
    std::memcpy(h, dp.reqs.data(), dp.reqs.size() * sizeof(DevDecodeReq));
    std::memcpy(h + dp.off_work, dp.work.data(), dp.work.size() * sizeof(DevDecodeWork));
    if (npage_ids) std::memcpy(h + dp.off_pages, p->page_ids, (size_t)npage_ids * sizeof(int32_t));
    std::memcpy(h + dp.off_tokreq, dp.tok_req.data(), dp.tok_req.size() * sizeof(int32_t));
  });
  if (s != CAS_OK) return s;
  DecodeParams kp{};
  kp.q = q;
  kp.k_pages = k_pages;
  kp.v_pages = v_pages;
  kp.o = o;
  kp.lse = lse;
  kp.reqs = (const DevDecodeReq *)ws;
  kp.work = (const DevDecodeWork *)(ws + dp.off_work);
  kp.page_ids = (const int32_t *)(ws + dp.off_pages);
  kp.tok_req = (const int32_t *)(ws + dp.off_tokreq);
  kp.part_lse = dp.max_split > 1 ? (float *)(ws + dp.off_plse) : nullptr;
  kp.part_o = dp.max_split > 1 ? (float *)(ws + dp.off_po) : nullptr;
  kp.plane = (int64_t)dp.Tq * dp.Hq;
  kp.Hkv = p->num_kv_heads;
  kp.g = p->group_size;
  kp.page_size = p->page_size;
  kp.Tq = dp.Tq;
  kp.scale_log2 = p->softmax_scale * 1.4426950408889634f;
  hipError_t e = timed("decode", stream, [&] { return launch_decode_bf16(kp, p->head_dim, (int)dp.work.size(), stream); });
  if (e != hipSuccess) return hip_fail("decode launch", e);
  if (dp.max_split > 1) {
    e = timed("decode_merge", stream, [&] { return launch_decode_merge_bf16(kp, p->head_dim, stream); });
    if (e != hipSuccess) return hip_fail("decode_merge launch", e);
  }
  return CAS_OK;
}

cas_status_t cas_cartridge_adam_workspace_size(const cas_adam_cartridge_t *carts, int32_t n,
                                               int32_t num_kv_heads, int32_t head_dim, size_t *bytes) {
  if (!bytes) return fail(CAS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  AdamPlan ap;
  cas_status_t s = build_adam(carts, n, num_kv_heads, head_dim, nullptr, ap);
  if (s != CAS_OK) return s;
  *bytes = ap.bytes;
  return CAS_OK;
}

cas_status_t cas_cartridge_adam(const cas_adam_cartridge_t *carts, int32_t n, int32_t num_kv_heads,
                                int32_t head_dim, const cas_adam_config_t *cfg, void *workspace,
                                size_t ws_bytes, void *hip_stream) {
  if (!cfg) return fail(CAS_ERR_INVALID_ARGUMENT, "cfg is NULL");
  AdamPlan ap;
  cas_status_t s = build_adam(carts, n, num_kv_heads, head_dim, cfg, ap);
  if (s != CAS_OK) return s;
  if (ap.chunks.empty()) return CAS_OK;
  s = check_workspace(workspace, ws_bytes, ap.bytes);
  if (s != CAS_OK) return s;
  hipStream_t stream = (hipStream_t)hip_stream;
  s = ring_upload(ap.bytes, workspace, stream, [&](char *h) {
    std::memcpy(h, ap.tensors.data(), ap.tensors.size() * sizeof(DevAdamT));
    std::memcpy(h + ap.off_chunks, ap.chunks.data(), ap.chunks.size() * sizeof(DevAdamChunk));
  });
  if (s != CAS_OK) return s;
  AdamParams p{};
  p.tensors = (const DevAdamT *)workspace;
  p.chunks = (const DevAdamChunk *)((char *)workspace + ap.off_chunks);
  p.Hkv = num_kv_heads;
  p.beta1 = cfg->beta1;
  p.beta2 = cfg->beta2;
  p.omb1 = 1.0f - cfg->beta1;
  p.omb2 = 1.0f - cfg->beta2;
  p.eps = cfg->eps;
  hipError_t e = timed("adam", stream, [&] { return launch_adam_bf16(p, head_dim, (int)ap.chunks.size(), stream); });
  if (e != hipSuccess) return hip_fail("adam launch", e);
  return CAS_OK;
}

cas_status_t cas_set_tuning(const cas_tuning_t *t) {
  if (!t) return fail(CAS_ERR_INVALID_ARGUMENT, "tuning is NULL");
  if (t->fwd_splits < 0 || t->dq_splits < 0 || t->fwd_splits > kMaxSplits || t->dq_splits > kMaxSplits)
    return fail(CAS_ERR_INVALID_ARGUMENT, "splits must be in [0, " + std::to_string(kMaxSplits) + "]");
  std::lock_guard<std::mutex> lk(g_tuning_mu);
  g_tuning = *t;
  return CAS_OK;
}

cas_status_t cas_get_tuning(cas_tuning_t *t) {
  if (!t) return fail(CAS_ERR_INVALID_ARGUMENT, "tuning is NULL");
  *t = tuning();
  return CAS_OK;
}

cas_status_t cas_prefix_attn_workspace_size(const cas_problem_t *p, int backward, size_t *bytes) {
  if (!bytes) return fail(CAS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  Plan pl;
  cas_status_t s = build_plan(p, backward != 0, pl);
  if (s != CAS_OK) return s;
  *bytes = backward ? pl.ws_bwd : pl.ws_fwd;
  return CAS_OK;
}

cas_status_t cas_plan_info(const cas_problem_t *p, cas_plan_info_t *out) {
  if (!out) return fail(CAS_ERR_INVALID_ARGUMENT, "out is NULL");
  Plan pf, pb;
  cas_status_t s = build_plan(p, false, pf);
  if (s != CAS_OK) return s;
  s = build_plan(p, true, pb);
  if (s != CAS_OK) return s;
  out->fwd_splits = pf.fwd_splits;
  out->dq_splits = pb.dq_splits;
  out->fwd_workgroups = pf.dt == kBF16 ? (int32_t)pf.items.size() : pf.nqblk_fwd * pf.Hkv * pf.B * pf.fwd_splits;
  out->dkdv_workgroups = (int32_t)pb.order_cap;
  out->unique_segments = (int32_t)pb.carts.size();
  out->total_key_tiles = (int32_t)(pb.order_cap / pb.Hkv);
  out->max_prefix_len = pf.max_prefix;
  out->ws_fwd_bytes = pf.ws_fwd;
  out->ws_bwd_bytes = pb.ws_bwd;
  return CAS_OK;
}

cas_status_t cas_prefix_attn_fwd(const cas_problem_t *p, const void *q, const void *k_self,
                                 const void *v_self, void *o, float *lse, void *workspace,
                                 size_t ws_bytes, void *hip_stream) {
  return prefix_attn_fwd_run(p, q, k_self, v_self, o, lse, workspace, ws_bytes, (hipStream_t)hip_stream,
                             nullptr);
}

cas_status_t cas_prefix_attn_bwd(const cas_problem_t *p, const void *q, const void *k_self,
                                 const void *v_self, const void *o, const float *lse,
                                 const void *d_o, void *dq, void *dk_self, void *dv_self,
                                 void *workspace, size_t ws_bytes, void *hip_stream) {
  Plan pl;
  cas_status_t s = build_plan(p, true, pl);
  if (s != CAS_OK) return s;
  if (!q || !k_self || !v_self || !o || !lse || !d_o)
    return fail(CAS_ERR_INVALID_ARGUMENT, "q, k_self, v_self, o, lse and d_o must be non-NULL");
  if (!aligned16(q) || !aligned16(k_self) || !aligned16(v_self) || !aligned16(o) || !aligned16(d_o) ||
      !aligned16(dq) || !aligned16(dk_self) || !aligned16(dv_self) || ((uintptr_t)lse & 3u))
    return fail(CAS_ERR_ALIGNMENT, "tensors must be 16-byte aligned (lse 4-byte)");
  const uintptr_t qbytes = (uintptr_t)pl.T * pl.Hq * pl.D * pl.esize;
  const uintptr_t kvbytes = (uintptr_t)pl.T * pl.Hkv * pl.D * pl.esize;
  std::vector<Interval> iv;
  iv.push_back({(uintptr_t)q, (uintptr_t)q + qbytes, false, 0, "q"});
  iv.push_back({(uintptr_t)k_self, (uintptr_t)k_self + kvbytes, false, 0, "k_self"});
  iv.push_back({(uintptr_t)v_self, (uintptr_t)v_self + kvbytes, false, 0, "v_self"});
  iv.push_back({(uintptr_t)o, (uintptr_t)o + qbytes, false, 0, "o"});
  iv.push_back({(uintptr_t)lse, (uintptr_t)lse + (uintptr_t)pl.T * pl.Hq * 4, false, 0, "lse"});
  iv.push_back({(uintptr_t)d_o, (uintptr_t)d_o + qbytes, false, 0, "d_o"});
  if (dq) iv.push_back({(uintptr_t)dq, (uintptr_t)dq + qbytes, true, (uintptr_t)dq, "dq"});
  if (dk_self) iv.push_back({(uintptr_t)dk_self, (uintptr_t)dk_self + kvbytes, true, (uintptr_t)dk_self, "dk_self"});
  if (dv_self) iv.push_back({(uintptr_t)dv_self, (uintptr_t)dv_self + kvbytes, true, (uintptr_t)dv_self, "dv_self"});
  add_segment_intervals(pl, p, true, iv);
  std::string msg;
  if (!overlap_free(iv, msg)) return fail(CAS_ERR_INVALID_ARGUMENT, msg);
  s = check_workspace(workspace, ws_bytes, pl.ws_bwd);
  if (s != CAS_OK) return s;

  hipStream_t stream = (hipStream_t)hip_stream;
  bind_self_tiles(pl, k_self, v_self);
  build_dkdv_order(pl, dk_self || dv_self);
  s = upload_tables(pl, true, workspace, stream);
  if (s != CAS_OK) return s;
  char *ws = (char *)workspace;
  float *nd = (float *)(ws + pl.off_nd);
  float *lse2 = (float *)(ws + pl.off_lse2);
  const float scale_log2 = pl.scale * 1.4426950408889634f;

  PreParams pp{};
  pp.o = o;
  pp.d_o = d_o;
  pp.lse = lse;
  pp.nd = nd;
  pp.lse2 = lse2;
  pp.rows = (const DevRow *)(ws + pl.off_rows);
  pp.B = pl.B;
  pp.Hkv = pl.Hkv;
  pp.g = pl.g;
  pp.nrows_max = pl.nrows_max;
  pp.nqb_max = pl.nqb_max;
  pp.lse_hs = pl.packed ? (int32_t)pl.T : pl.Sq;
  pp.q = q;
  pp.qT = pl.dt == kBF16 ? ws + pl.off_qT : nullptr;
  pp.doT = pl.dt == kBF16 ? ws + pl.off_doT : nullptr;
  // bf16: the statistics and the transposed Q / dO blocks in one pass.
  hipError_t e = timed("bwd_pre", stream, [&] {
    return pl.dt == kBF16 ? launch_bwd_prologue_bf16(pp, pl.D, stream) : launch_bwd_pre(pp, pl.dt, pl.D, stream);
  });
  if (e != hipSuccess) return hip_fail("bwd_pre launch", e);

  const int n_wg = (int)pl.dkdv_grid;
  auto run_dq = [&]() -> hipError_t {
    if (!dq) return hipSuccess;
    DqParams dp{};
    dp.q = q;
    dp.k_self = k_self;
    dp.v_self = v_self;
    dp.d_o = d_o;
    dp.nd = nd;
    dp.lse2 = lse2;
    dp.dq = dq;
    dp.part_dq = pl.dq_splits > 1 ? (float *)(ws + pl.off_part_dq) : nullptr;
    dp.segs = (const DevSeg *)(ws + pl.off_segs);
    dp.tiles = (const DevTile *)(ws + pl.off_tiles);
    dp.items = (const DevItem *)(ws + pl.off_items);
    dp.rows = (const DevRow *)(ws + pl.off_rows);
    dp.plane = pl.T * pl.Hq;
    dp.B = pl.B;
    dp.Smax = pl.Smax;
    dp.Hkv = pl.Hkv;
    dp.g = pl.g;
    dp.nrows_max = pl.nrows_max;
    dp.nqblk = pl.nqblk_dq;
    dp.splits = pl.dq_splits;
    dp.n_items = (int32_t)pl.items.size();
    dp.scale_log2 = scale_log2;
    dp.scale = pl.scale;
    hipError_t r = timed("dq", stream, [&] { return launch_dq(dp, pl.dt, pl.D, stream); });
    if (r != hipSuccess || pl.dq_splits <= 1) return r;
    DqReduceParams rp{};
    rp.part_dq = dp.part_dq;
    rp.dq = dq;
    rp.rows = dp.rows;
    rp.plane = dp.plane;
    rp.B = pl.B;
    rp.Hkv = pl.Hkv;
    rp.g = pl.g;
    rp.nrows_max = pl.nrows_max;
    rp.splits = pl.dq_splits;
    rp.scale = pl.scale;
    return timed("dq_reduce", stream, [&] { return launch_dq_reduce(rp, pl.dt, pl.D, stream); });
  };
  if (n_wg > 0) {
    DkdvParams kp{};
    kp.q = q;
    kp.k_self = k_self;
    kp.v_self = v_self;
    kp.d_o = d_o;
    kp.nd = nd;
    kp.lse2 = lse2;
    kp.qT = pp.qT;
    kp.doT = pp.doT;
    kp.dk_self = dk_self;
    kp.dv_self = dv_self;
    kp.carts = (const DevCart *)(ws + pl.off_carts);
    kp.uses = (const int32_t *)(ws + pl.off_uses);
    kp.rows = pp.rows;
    kp.order = (const DevWg *)(ws + pl.off_order);
    kp.queues = pl.queues.empty() ? nullptr : (const DevQueue *)(ws + pl.off_queues);
    kp.claim = pl.queues.empty() ? nullptr : (int32_t *)(ws + pl.off_claim);
    kp.xcds = pl.xcds;
    kp.n_carts = (int32_t)pl.carts.size();
    kp.cart_tiles = pl.cart_tiles;
    kp.self_tiles = std::max(pl.self_tiles_max, 1);
    kp.B = pl.B;
    kp.Hkv = pl.Hkv;
    kp.g = pl.g;
    kp.scale_log2 = scale_log2;
    kp.scale = pl.scale;
    e = timed("dkdv", stream, [&] { return launch_dkdv(kp, pl.dt, pl.D, n_wg, stream); });
    if (e != hipSuccess) return hip_fail("dkdv launch", e);
  }
  e = run_dq();
  if (e != hipSuccess) return hip_fail("dq launch", e);
  return CAS_OK;
}

cas_status_t cas_cartridge_stage(const cas_stage_copy_t *copies, int32_t n, void *side_stream,
                                 void *done_event) {
  if (n < 0) return fail(CAS_ERR_INVALID_ARGUMENT, "n must be >= 0");
  if (n > 0 && !copies) return fail(CAS_ERR_INVALID_ARGUMENT, "copies is NULL");
  for (int i = 0; i < n; ++i) {
    if (copies[i].bytes == 0) continue;
    if (!copies[i].host_src || !copies[i].dev_dst)
      return fail(CAS_ERR_INVALID_ARGUMENT, "copy " + std::to_string(i) + ": NULL pointer");
  }
  for (int i = 0; i < n; ++i) {
    const cas_stage_copy_t &c = copies[i];
    if (c.bytes == 0) continue;
    const void *ends[2] = {c.host_src, (const char *)c.host_src + c.bytes - 1};
    for (const void *ptr : ends) {
      hipPointerAttribute_t a;
      hipError_t e = hipPointerGetAttributes(&a, ptr);
      if (e != hipSuccess || a.type != hipMemoryTypeHost) {
        (void)hipGetLastError();
        return fail(CAS_ERR_NOT_PINNED, "copy " + std::to_string(i) + ": host_src is not pinned host memory");
      }
    }
    hipPointerAttribute_t d;
    hipError_t e = hipPointerGetAttributes(&d, c.dev_dst);
    if (e != hipSuccess || d.type != hipMemoryTypeDevice) {
      (void)hipGetLastError();
      return fail(CAS_ERR_INVALID_ARGUMENT, "copy " + std::to_string(i) + ": dev_dst is not device memory");
    }
  }
  std::vector<HostCopy> list((size_t)n);
  for (int i = 0; i < n; ++i) list[i] = {copies[i].host_src, copies[i].dev_dst, copies[i].bytes};
  hipStream_t s = (hipStream_t)side_stream;
  {
    hipError_t e = enqueue_copies(list.data(), n, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail("hipMemcpyAsync", e);
  }
  if (done_event) {
    hipError_t e = hipEventRecord((hipEvent_t)done_event, s);
    if (e != hipSuccess) return hip_fail("hipEventRecord", e);
  }
  return CAS_OK;
}

cas_status_t cas_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_time_mu);
  g_timing = enable != 0;
  return CAS_OK;
}

cas_status_t cas_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_time_mu);
  for (auto &t : g_pending) {
    (void)hipEventSynchronize(t.b);
    g_event_pool.push_back(t.a);
    g_event_pool.push_back(t.b);
  }
  g_pending.clear();
  g_totals.clear();
  return CAS_OK;
}

cas_status_t cas_timing_read(cas_kernel_time_t *out, int32_t cap, int32_t *n_out) {
  if (!n_out || (cap > 0 && !out)) return fail(CAS_ERR_INVALID_ARGUMENT, "NULL output");
  std::lock_guard<std::mutex> lk(g_time_mu);
  for (auto &t : g_pending) {
    hipError_t e = hipEventSynchronize(t.b);
    if (e != hipSuccess) return hip_fail("hipEventSynchronize", e);
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, t.a, t.b);
    if (e != hipSuccess) return hip_fail("hipEventElapsedTime", e);
    auto &acc = g_totals[t.name];
    acc.first += 1;
    acc.second += ms;
    g_event_pool.push_back(t.a);
    g_event_pool.push_back(t.b);
  }
  g_pending.clear();
  int32_t i = 0;
  for (auto &kv : g_totals) {
    if (i < cap) {
      std::memset(out[i].name, 0, sizeof(out[i].name));
      std::strncpy(out[i].name, kv.first.c_str(), sizeof(out[i].name) - 1);
      out[i].launches = kv.second.first;
      out[i].total_ms = kv.second.second;
    }
    ++i;
  }
  *n_out = i;
  return CAS_OK;
}

}  // extern "C"
