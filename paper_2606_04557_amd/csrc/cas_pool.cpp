// libcas budget manager: a pool of N cartridges of which B train on the GPU
// at a time, rotated every R optimizer steps (least-trained first), with the
// fp32 Adam moments of the offloaded cartridges in pinned host memory or in a
// file on a local (NVMe) file system.
//
// Copies between host and GPU run on the pool's own stream. The file tier's
// transfers of a rotation run on threads of their own, overlapped with the
// training steps: a rotation's reads until the next rotation, its writes
// (double-buffered) until the one after.
#include <hip/hip_runtime.h>

#include <fcntl.h>
#include <sys/types.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <cmath>
#include <cstring>
#include <functional>
#include <future>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/cas.h"
#include "cas_host.h"

using namespace cas;

namespace {

size_t align_to(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Evict the n active cartridges with the most steps, admit the n offloaded
// ones with the fewest (ties: lower id), n = min(floor(phi * B), offloaded).
int plan_rotation(const int32_t *steps, const uint8_t *active, int N, int B, float phi, int32_t *evict,
                  int32_t *admit) {
  std::vector<int> act, off;
  for (int c = 0; c < N; ++c) (active[c] ? act : off).push_back(c);
  const int n = std::min<int>((int)std::floor((double)phi * B + 1e-9), (int)off.size());
  std::stable_sort(act.begin(), act.end(), [&](int a, int b) { return steps[a] > steps[b]; });
  std::stable_sort(off.begin(), off.end(), [&](int a, int b) { return steps[a] < steps[b]; });
  const int m = std::min<int>(n, (int)act.size());
  for (int i = 0; i < m; ++i) {
    if (evict) evict[i] = act[i];
    if (admit) admit[i] = off[i];
  }
  return m;
}

// Whole-buffer positioned file transfers (short transfers and interrupts
// are retried). "" on success, else a message.
std::string pread_all(int fd, void *buf, size_t n, off_t off) {
  char *p = (char *)buf;
  while (n) {
    const ssize_t r = pread(fd, p, n, off);
    if (r < 0 && errno == EINTR) continue;
    if (r < 0) return std::string("moment file read: ") + std::strerror(errno);
    if (r == 0) return "moment file read: unexpected end of file";
    p += r;
    n -= (size_t)r;
    off += r;
  }
  return "";
}

std::string pwrite_all(int fd, const void *buf, size_t n, off_t off) {
  const char *p = (const char *)buf;
  while (n) {
    const ssize_t r = pwrite(fd, p, n, off);
    if (r < 0 && errno == EINTR) continue;
    if (r < 0) return std::string("moment file write: ") + std::strerror(errno);
    p += r;
    n -= (size_t)r;
    off += r;
  }
  return "";
}

// Runs f(0) .. f(n-1) on up to kIoThreads threads (file transfers of
// separate pieces proceed in parallel: more requests in flight for the
// drive, several cores for page-cache copies); returns the first error.
constexpr int kIoThreads = 4;
std::string parallel_io(int n, const std::function<std::string(int)> &f) {
  std::atomic<int> next{0};
  std::mutex mu;
  std::string err;
  auto run = [&]() {
    for (int i; (i = next++) < n;) {
      std::string e = f(i);
      if (!e.empty()) {
        std::lock_guard<std::mutex> lk(mu);
        if (err.empty()) err = e;
      }
    }
  };
  std::vector<std::thread> th;
  for (int t = 1; t < std::min(n, kIoThreads); ++t) {
    try {
      th.emplace_back(run);
    } catch (...) {
      break;   // fewer threads: the pieces still all run
    }
  }
  run();
  for (auto &t : th) t.join();
  return err;
}

}  // namespace

struct cas_pool {
  int N = 0, Hkv = 0, D = 0, B = 0, R = 1, S = 0, frozen = 0, device = 0;
  float phi = 0.0f;
  std::vector<int64_t> lens;
  int64_t max_len = 0, tok_el = 0;
  // Pinned host tier: per cartridge K, V (bf16), then, without the file
  // tier, its moments m1_k, m2_k, m1_v, m2_v (fp32).
  char *host = nullptr;
  std::vector<size_t> hoff;
  // Device slots: K, V, dK, dV (A bytes each), four moments (M bytes each).
  char *dev = nullptr;
  size_t A = 0, M = 0, slot_bytes = 0;
  // File tier: the moments of cartridge c at foff[c], laid out as in the
  // host tier; pinned moment buffers (mbuf_bytes each): two sets of nbuf for
  // evictions (used by alternate rotations), one set of nbuf for admissions.
  int fd = -1;
  std::vector<off_t> foff;
  char *mbuf = nullptr;
  int nbuf = 0;
  size_t mbuf_bytes = 0;
  // The file tier's transfers, each on a thread of its own: the writes of
  // the evicted moments out of eviction set w (io_write[w], cartridges
  // io_written[w]) and the reads of the next admissions' moments (io_read;
  // after any pending write of one of its cartridges). io_err keeps the
  // first failure.
  std::shared_future<std::string> io_write[2], io_read;
  std::vector<int32_t> io_written[2];
  int wset = 0;   // eviction set of the next eviction
  std::string io_err;
  std::vector<int32_t> steps, slot_cart, active, staging, next_admit;   // slot_cart: cartridge in each slot or -1
  int64_t step_count = 0;
  bool loaded = false;
  hipStream_t side = nullptr;
  hipEvent_t ev_compute = nullptr, ev_admit = nullptr, ev_evict[2] = {nullptr, nullptr};

  bool file() const { return fd >= 0; }
  size_t kv_bytes(int c) const { return (size_t)lens[c] * tok_el * 2; }
  size_t mom_bytes(int c) const { return (size_t)lens[c] * tok_el * 4; }
  char *slot_ptr(int slot, int part) const {   // 0 K, 1 V, 2 dK, 3 dV, 4.. moments m1k, m2k, m1v, m2v
    char *b = dev + (size_t)slot * slot_bytes;
    return part < 4 ? b + part * A : b + 4 * A + (part - 4) * M;
  }
  char *host_kv(int c, int part) const { return host + hoff[c] + part * kv_bytes(c); }   // 0 K, 1 V
  char *host_moments(int c) const { return file() ? nullptr : host + hoff[c] + 2 * kv_bytes(c); }
  char *evict_buf(int set, int i) const { return mbuf + (size_t)(set * nbuf + i) * mbuf_bytes; }
  char *admit_buf(int i) const { return mbuf + (size_t)(2 * nbuf + i) * mbuf_bytes; }

  // Copies of cartridge c's K/V and moments between host memory (moments at
  // hm: the host tier or a pinned buffer of the file tier) and slot.
  void copies(int c, int slot, const char *hm, bool to_device, std::vector<HostCopy> &out) const {
    auto add = [&](const char *h, char *d, size_t n) {
      if (to_device) out.push_back({h, d, n});
      else out.push_back({d, (void *)h, n});
    };
    add(host_kv(c, 0), slot_ptr(slot, 0), kv_bytes(c));
    add(host_kv(c, 1), slot_ptr(slot, 1), kv_bytes(c));
    for (int i = 0; i < 4; ++i) add(hm + i * mom_bytes(c), slot_ptr(slot, 4 + i), mom_bytes(c));
  }

  // Moment pieces of a transfer list: (list index, moment tensor), one file
  // transfer each.
  template <typename F>
  std::string moment_pieces(const std::vector<int32_t> &cs, F &&f) {
    return parallel_io(4 * (int)cs.size(), [&](int k) { return f(k / 4, k % 4); });
  }

  // Brings cartridges cs[i] into slots sl[i] on the pool's stream and records
  // ev_admit after them. With the file tier this runs on a thread of its own:
  // it waits for the previous admission's copies out of the admission
  // buffers (and, for a cartridge written by the running eviction, for that
  // write), reads the moments from the file into the buffers and only then
  // enqueues the copies; the caller must join it (io_check) before it waits
  // on ev_admit.
  hipError_t admit(const std::vector<int32_t> &cs, const std::vector<int32_t> &sl) {
    if (!file()) {
      std::vector<HostCopy> list;
      for (size_t i = 0; i < cs.size(); ++i) copies(cs[i], sl[i], host_moments(cs[i]), true, list);
      hipError_t e = enqueue_copies(list.data(), (int)list.size(), hipMemcpyHostToDevice, side);
      return e == hipSuccess ? hipEventRecord(ev_admit, side) : e;
    }
    std::vector<std::shared_future<std::string>> wr;   // pending writes of these cartridges
    for (int w = 0; w < 2; ++w) {
      bool hit = false;
      for (int c : cs) hit |= std::find(io_written[w].begin(), io_written[w].end(), c) != io_written[w].end();
      if (hit && io_write[w].valid()) wr.push_back(io_write[w]);
    }
    auto task = [this, cs, sl, wr]() -> std::string {
      (void)hipSetDevice(device);
      for (const auto &f : wr)
        if (!f.get().empty()) return "";   // the write's error is reported on its own
      hipError_t e = hipEventSynchronize(ev_admit);
      if (e != hipSuccess) return std::string("hipEventSynchronize: ") + hipGetErrorString(e);
      std::string r = moment_pieces(cs, [&](int i, int part) {
        const size_t m = mom_bytes(cs[i]);
        return pread_all(fd, admit_buf(i) + part * m, m, foff[cs[i]] + (off_t)(part * m));
      });
      if (!r.empty()) return r;
      std::vector<HostCopy> list;
      for (size_t i = 0; i < cs.size(); ++i) copies(cs[i], sl[i], admit_buf((int)i), true, list);
      e = enqueue_copies(list.data(), (int)list.size(), hipMemcpyHostToDevice, side);
      if (e == hipSuccess) e = hipEventRecord(ev_admit, side);
      return e == hipSuccess ? std::string() : std::string("admission copies: ") + hipGetErrorString(e);
    };
    return launch(io_read, task);
  }

  // Starts task on a thread of its own, its result in f.
  template <typename T>
  hipError_t launch(std::shared_future<std::string> &f, T &&task) {
    try {
      f = std::async(std::launch::async, std::forward<T>(task)).share();
    } catch (...) {
      return hipErrorOutOfMemory;   // no thread could be started
    }
    return hipSuccess;
  }

  // Copies cartridges cs[i] out of slots sl[i] on the pool's stream (after
  // whatever it already holds). With the file tier at most nbuf at a time:
  // their moments land in the next eviction set (after the write that last
  // used it has finished) and a thread of its own writes them to the file
  // once the set's event has passed.
  hipError_t evict(const std::vector<int32_t> &cs, const std::vector<int32_t> &sl) {
    const int w = wset;
    if (file()) {
      join(io_write[w]);
      if (!io_err.empty()) return hipErrorUnknown;   // reported by the caller's io_check
    }
    std::vector<HostCopy> list;
    for (size_t i = 0; i < cs.size(); ++i)
      copies(cs[i], sl[i], file() ? evict_buf(w, (int)i) : host_moments(cs[i]), false, list);
    hipError_t e = enqueue_copies(list.data(), (int)list.size(), hipMemcpyDeviceToHost, side);
    if (e != hipSuccess || !file()) return e;
    e = hipEventRecord(ev_evict[w], side);
    if (e != hipSuccess) return e;
    io_written[w] = cs;
    wset ^= 1;
    return launch(io_write[w], [this, cs, w]() -> std::string {
      (void)hipSetDevice(device);
      hipError_t e2 = hipEventSynchronize(ev_evict[w]);
      if (e2 != hipSuccess) return std::string("hipEventSynchronize: ") + hipGetErrorString(e2);
      return moment_pieces(cs, [&](int i, int part) {
        const size_t m = mom_bytes(cs[i]);
        return pwrite_all(fd, evict_buf(w, i) + part * m, m, foff[cs[i]] + (off_t)(part * m));
      });
    });
  }

  // Plans and starts the next admissions into the staging slots.
  hipError_t prefetch() {
    std::vector<uint8_t> act(N, 0);
    for (int sl : active) act[slot_cart[sl]] = 1;
    next_admit.assign(S, -1);
    const int n = plan_rotation(steps.data(), act.data(), N, B, phi, nullptr, next_admit.data());
    next_admit.resize(n);
    std::vector<int32_t> sl(staging.begin(), staging.begin() + n);
    for (int i = 0; i < n; ++i) slot_cart[sl[i]] = next_admit[i];
    return admit(next_admit, sl);
  }

  // Waits for one transfer; its failure goes to io_err.
  void join(std::shared_future<std::string> &f) {
    if (!f.valid()) return;
    std::string e;
    try {
      e = f.get();
    } catch (const std::exception &x) {
      e = std::string("moment file transfer: ") + x.what();
    }
    if (io_err.empty()) io_err = e;
    f = std::shared_future<std::string>();
  }

  // Joins the admission reads (all = true: every transfer); CAS_ERR_IO after
  // any failure.
  cas_status_t io_check(bool all = false) {
    join(io_read);
    if (all)
      for (int w = 0; w < 2; ++w) {
        join(io_write[w]);
        io_written[w].clear();
      }
    return io_err.empty() ? CAS_OK : set_error(CAS_ERR_IO, io_err);
  }

  void release() {
    (void)io_check(true);
    if (side) (void)hipStreamSynchronize(side);
    if (side) (void)hipStreamDestroy(side);
    if (ev_compute) (void)hipEventDestroy(ev_compute);
    if (ev_admit) (void)hipEventDestroy(ev_admit);
    for (hipEvent_t &x : ev_evict)
      if (x) (void)hipEventDestroy(x);
    if (dev) (void)hipFree(dev);
    if (host) (void)hipHostFree(host);
    if (mbuf) (void)hipHostFree(mbuf);
    if (fd >= 0) close(fd);
    side = nullptr;
    ev_compute = ev_admit = ev_evict[0] = ev_evict[1] = nullptr;
    dev = host = mbuf = nullptr;
    fd = -1;
  }
};

extern "C" {

cas_status_t cas_pool_plan_rotation(const int32_t *steps, const uint8_t *active, int32_t n, int32_t budget,
                                    float swap_fraction, int32_t *evict, int32_t *admit, int32_t *n_swap) {
  if (!steps || !active || !n_swap || n < 1 || budget < 1 || !(swap_fraction >= 0.0f && swap_fraction <= 1.0f))
    return set_error(CAS_ERR_INVALID_ARGUMENT, "bad rotation query");
  *n_swap = plan_rotation(steps, active, n, budget, swap_fraction, evict, admit);
  return CAS_OK;
}

cas_status_t cas_pool_create(const cas_pool_config_t *cfg, cas_pool_t **out) {
  if (!cfg || !out) return set_error(CAS_ERR_INVALID_ARGUMENT, "cfg or out is NULL");
  *out = nullptr;
  if (cfg->num_cartridges < 1 || !cfg->lens)
    return set_error(CAS_ERR_INVALID_ARGUMENT, "need >= 1 cartridge and lens");
  if (cfg->num_kv_heads < 1) return set_error(CAS_ERR_INVALID_ARGUMENT, "num_kv_heads must be >= 1");
  if (cfg->head_dim != 64 && cfg->head_dim != 128)
    return set_error(CAS_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (cfg->budget < 1 || cfg->budget > cfg->num_cartridges)
    return set_error(CAS_ERR_INVALID_ARGUMENT, "budget must lie in [1, num_cartridges]");
  if (cfg->rotate_every < 1 || !(cfg->swap_fraction >= 0.0f && cfg->swap_fraction <= 1.0f) ||
      cfg->frozen_tokens < 0)
    return set_error(CAS_ERR_INVALID_ARGUMENT, "rotate_every >= 1, swap_fraction in [0, 1], frozen_tokens >= 0");
  std::unique_ptr<cas_pool> p(new cas_pool());
  p->N = cfg->num_cartridges;
  p->Hkv = cfg->num_kv_heads;
  p->D = cfg->head_dim;
  p->B = cfg->budget;
  p->R = cfg->rotate_every;
  p->phi = cfg->swap_fraction;
  p->frozen = cfg->frozen_tokens;
  p->tok_el = (int64_t)p->Hkv * p->D;
  p->S = std::min<int>((int)std::floor((double)p->phi * p->B + 1e-9), p->N - p->B);
  for (int c = 0; c < p->N; ++c) {
    const int64_t L = cfg->lens[c];
    if (L < 1 || L > (1 << 30))
      return set_error(CAS_ERR_INVALID_ARGUMENT, "cartridge lengths must lie in [1, 2^30]");
    p->lens.push_back(L);
    p->max_len = std::max(p->max_len, L);
  }
  // The moment file first: its errors need no device.
  if (cfg->moment_dir) {
    std::string path = std::string(cfg->moment_dir) + "/cas_moments_XXXXXX";
    std::vector<char> name(path.begin(), path.end());
    name.push_back('\0');
    const int fd = mkstemp(name.data());
    if (fd < 0)
      return set_error(CAS_ERR_IO, "moment file in " + std::string(cfg->moment_dir) + ": " + std::strerror(errno));
    unlink(name.data());   // unnamed from now on: gone when closed or at process end
    p->fd = fd;
    off_t off = 0;
    for (int c = 0; c < p->N; ++c) {
      p->foff.push_back(off);
      off += (off_t)align_to(4 * p->mom_bytes(c), 4096);
    }
    // Zero moments, as for a new cartridge; the blocks are reserved now so
    // that no write has to allocate them.
    const int r = off ? posix_fallocate(fd, 0, off) : 0;
    if (r != 0 && ftruncate(fd, off) != 0) {
      const std::string msg = std::string("moment file size: ") + std::strerror(errno);
      p->release();
      return set_error(CAS_ERR_IO, msg);
    }
  }
  size_t hb = 0;
  for (int c = 0; c < p->N; ++c) {
    p->hoff.push_back(hb);
    hb += align_to(2 * p->kv_bytes(c) + (p->file() ? 0 : 4 * p->mom_bytes(c)), 256);
  }
  p->A = align_to((size_t)p->max_len * p->tok_el * 2, 256);
  p->M = align_to((size_t)p->max_len * p->tok_el * 4, 256);
  p->slot_bytes = 4 * p->A + 4 * p->M;
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) {
    p->release();
    return set_hip_error("hipGetDevice", e);
  }
  e = hipHostMalloc((void **)&p->host, hb, hipHostMallocDefault);
  if (e != hipSuccess) {
    p->host = nullptr;
    p->release();
    return set_hip_error("hipHostMalloc", e);
  }
  std::memset(p->host, 0, hb);
  if (p->file()) {
    p->nbuf = std::max(p->S, 1);
    p->mbuf_bytes = align_to(4 * (size_t)p->max_len * p->tok_el * 4, 4096);
    e = hipHostMalloc((void **)&p->mbuf, 3 * (size_t)p->nbuf * p->mbuf_bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
      p->mbuf = nullptr;
      p->release();
      return set_hip_error("hipHostMalloc (moment buffers)", e);
    }
  }
  e = hipMalloc((void **)&p->dev, p->slot_bytes * (size_t)(p->B + p->S));
  if (e != hipSuccess) {
    p->dev = nullptr;
    p->release();
    return set_hip_error("hipMalloc", e);
  }
  if ((e = hipStreamCreateWithFlags(&p->side, hipStreamNonBlocking)) != hipSuccess ||
      (e = hipEventCreateWithFlags(&p->ev_compute, hipEventDisableTiming)) != hipSuccess ||
      (e = hipEventCreateWithFlags(&p->ev_admit, hipEventDisableTiming)) != hipSuccess ||
      (e = hipEventCreateWithFlags(&p->ev_evict[0], hipEventDisableTiming)) != hipSuccess ||
      (e = hipEventCreateWithFlags(&p->ev_evict[1], hipEventDisableTiming)) != hipSuccess) {
    p->release();
    return set_hip_error("pool stream/event", e);
  }
  p->steps.assign(p->N, 0);
  p->slot_cart.assign(p->B + p->S, -1);
  *out = p.release();
  return CAS_OK;
}

cas_status_t cas_pool_destroy(cas_pool_t *p) {
  if (!p) return CAS_OK;
  p->release();
  delete p;
  return CAS_OK;
}

cas_status_t cas_pool_host_cartridge(cas_pool_t *p, int32_t c, cas_adam_cartridge_t *v) {
  if (!p || !v || c < 0 || c >= p->N) return set_error(CAS_ERR_INVALID_ARGUMENT, "bad pool, view or cartridge");
  *v = cas_adam_cartridge_t{};
  v->k = p->host_kv(c, 0);
  v->v = p->host_kv(c, 1);
  if (char *m = p->host_moments(c)) {
    v->m1_k = (float *)m;
    v->m2_k = (float *)(m + p->mom_bytes(c));
    v->m1_v = (float *)(m + 2 * p->mom_bytes(c));
    v->m2_v = (float *)(m + 3 * p->mom_bytes(c));
  }
  v->len = p->lens[c];
  v->stride_tok = p->tok_el;
  v->stride_head = p->D;
  v->step = p->steps[c];
  v->frozen_tokens = p->frozen;
  return CAS_OK;
}

cas_status_t cas_pool_read_moments(cas_pool_t *p, int32_t c, float *dst) {
  if (!p || !dst || c < 0 || c >= p->N) return set_error(CAS_ERR_INVALID_ARGUMENT, "bad pool, cartridge or dst");
  cas_status_t s = p->io_check(true);
  if (s != CAS_OK) return s;
  const size_t n = 4 * p->mom_bytes(c);
  if (!p->file()) {
    std::memcpy(dst, p->host_moments(c), n);
    return CAS_OK;
  }
  const std::string r = pread_all(p->fd, dst, n, p->foff[c]);
  return r.empty() ? CAS_OK : set_error(CAS_ERR_IO, r);
}

cas_status_t cas_pool_load(cas_pool_t *p, void *compute_stream) {
  if (!p) return set_error(CAS_ERR_INVALID_ARGUMENT, "pool is NULL");
  if (p->loaded) return set_error(CAS_ERR_INVALID_ARGUMENT, "pool already loaded");
  // Active set: the B least-trained cartridges (ties: lower id).
  std::vector<int> order(p->N);
  for (int c = 0; c < p->N; ++c) order[c] = c;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return p->steps[a] < p->steps[b]; });
  p->active.clear();
  p->staging.clear();
  for (int i = 0; i < p->B; ++i) {
    p->slot_cart[i] = order[i];
    p->active.push_back(i);
  }
  for (int i = 0; i < p->S; ++i) p->staging.push_back(p->B + i);
  hipError_t e = hipSuccess;
  if (!p->file()) {
    std::vector<HostCopy> list;
    for (int i = 0; i < p->B; ++i) p->copies(order[i], i, p->host_moments(order[i]), true, list);
    e = enqueue_copies(list.data(), (int)list.size(), hipMemcpyHostToDevice, p->side);
  } else {
    // Through the admission buffers, nbuf cartridges at a time.
    for (int i0 = 0; i0 < p->B && e == hipSuccess; i0 += p->nbuf) {
      std::vector<HostCopy> list;
      for (int i = i0; i < std::min(p->B, i0 + p->nbuf); ++i) {
        const std::string r = pread_all(p->fd, p->admit_buf(i - i0), 4 * p->mom_bytes(order[i]), p->foff[order[i]]);
        if (!r.empty()) return set_error(CAS_ERR_IO, r);
        p->copies(order[i], i, p->admit_buf(i - i0), true, list);
      }
      e = enqueue_copies(list.data(), (int)list.size(), hipMemcpyHostToDevice, p->side);
      if (e == hipSuccess) e = hipStreamSynchronize(p->side);
    }
  }
  if (e != hipSuccess) return set_hip_error("pool load", e);
  e = hipEventRecord(p->ev_compute, p->side);   // active set landed
  if (e != hipSuccess) return set_hip_error("hipEventRecord", e);
  e = hipStreamWaitEvent((hipStream_t)compute_stream, p->ev_compute, 0);
  if (e != hipSuccess) return set_hip_error("hipStreamWaitEvent", e);
  e = p->prefetch();
  if (e != hipSuccess) return set_hip_error("pool prefetch", e);
  p->loaded = true;
  return CAS_OK;
}

cas_status_t cas_pool_active(cas_pool_t *p, int32_t *cart_ids, cas_adam_cartridge_t *views, int32_t cap, int32_t *n) {
  if (!p || !n || !p->loaded) return set_error(CAS_ERR_INVALID_ARGUMENT, "pool is NULL or not loaded");
  *n = (int32_t)p->active.size();
  for (int i = 0; i < (int)p->active.size() && i < cap; ++i) {
    const int sl = p->active[i], c = p->slot_cart[sl];
    if (cart_ids) cart_ids[i] = c;
    if (!views) continue;
    cas_adam_cartridge_t &v = views[i];
    v = cas_adam_cartridge_t{};
    v.k = p->slot_ptr(sl, 0);
    v.v = p->slot_ptr(sl, 1);
    v.dk = p->slot_ptr(sl, 2);
    v.dv = p->slot_ptr(sl, 3);
    v.m1_k = (float *)p->slot_ptr(sl, 4);
    v.m2_k = (float *)p->slot_ptr(sl, 5);
    v.m1_v = (float *)p->slot_ptr(sl, 6);
    v.m2_v = (float *)p->slot_ptr(sl, 7);
    v.len = p->lens[c];
    v.stride_tok = p->tok_el;
    v.stride_head = p->D;
    v.step = p->steps[c];
    v.frozen_tokens = p->frozen;
  }
  return CAS_OK;
}

cas_status_t cas_pool_end_step(cas_pool_t *p, void *compute_stream) {
  if (!p || !p->loaded) return set_error(CAS_ERR_INVALID_ARGUMENT, "pool is NULL or not loaded");
  for (int sl : p->active) ++p->steps[p->slot_cart[sl]];
  ++p->step_count;
  if (p->S == 0 || p->step_count % p->R != 0) return CAS_OK;
  // The previous rotation's file reads are done and its admissions are
  // enqueued (ev_admit recorded).
  cas_status_t s = p->io_check();
  if (s != CAS_OK) return s;
  hipStream_t cs = (hipStream_t)compute_stream;
  std::vector<uint8_t> act(p->N, 0);
  for (int sl : p->active) act[p->slot_cart[sl]] = 1;
  std::vector<int32_t> ev(p->S);
  const int n = plan_rotation(p->steps.data(), act.data(), p->N, p->B, p->phi, ev.data(), nullptr);
  if (n != (int)p->next_admit.size()) return set_error(CAS_ERR_INVALID_ARGUMENT, "rotation size changed");
  ev.resize(n);
  // Evict after the compute stream's last use of the active set.
  hipError_t e = hipEventRecord(p->ev_compute, cs);
  if (e == hipSuccess) e = hipStreamWaitEvent(p->side, p->ev_compute, 0);
  if (e != hipSuccess) return set_hip_error("pool rotation sync", e);
  std::vector<int32_t> freed;
  for (int c : ev)
    for (int a : p->active)
      if (p->slot_cart[a] == c) freed.push_back(a);
  e = p->evict(ev, freed);
  if (e != hipSuccess) return p->io_err.empty() ? set_hip_error("pool eviction", e) : set_error(CAS_ERR_IO, p->io_err);
  for (int sl : freed) p->slot_cart[sl] = -1;
  // The prefetched cartridges join the active set once their copies landed.
  std::vector<int32_t> next_active;
  for (int a : p->active)
    if (std::find(freed.begin(), freed.end(), a) == freed.end()) next_active.push_back(a);
  for (int i = 0; i < n; ++i) next_active.push_back(p->staging[i]);
  e = hipStreamWaitEvent(cs, p->ev_admit, 0);
  if (e != hipSuccess) return set_hip_error("hipStreamWaitEvent", e);
  std::vector<int32_t> next_staging = freed;
  for (int i = n; i < (int)p->staging.size(); ++i) next_staging.push_back(p->staging[i]);
  p->active = next_active;
  p->staging = next_staging;
  e = p->prefetch();   // after the evictions on the pool's stream (and thread)
  if (e != hipSuccess) return set_hip_error("pool prefetch", e);
  return CAS_OK;
}

cas_status_t cas_pool_flush(cas_pool_t *p, void *compute_stream) {
  if (!p || !p->loaded) return set_error(CAS_ERR_INVALID_ARGUMENT, "pool is NULL or not loaded");
  cas_status_t s = p->io_check();
  if (s != CAS_OK) return s;
  hipError_t e = hipEventRecord(p->ev_compute, (hipStream_t)compute_stream);
  if (e == hipSuccess) e = hipStreamWaitEvent(p->side, p->ev_compute, 0);
  // With the file tier, nbuf cartridges at a time through the eviction sets.
  const int batch = p->file() ? p->nbuf : (int)p->active.size();
  for (size_t i0 = 0; i0 < p->active.size() && e == hipSuccess; i0 += batch) {
    std::vector<int32_t> cs, sl;
    for (size_t i = i0; i < std::min(p->active.size(), i0 + batch); ++i) {
      sl.push_back(p->active[i]);
      cs.push_back(p->slot_cart[p->active[i]]);
    }
    e = p->evict(cs, sl);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(p->side);
  s = p->io_check(true);
  if (s != CAS_OK) return s;
  if (e != hipSuccess) return set_hip_error("pool flush", e);
  return CAS_OK;
}

}  // extern "C"
