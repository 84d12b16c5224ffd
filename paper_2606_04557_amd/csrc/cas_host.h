// Host-side helpers shared by libcas's host sources (no device code).
#pragma once

#include <hip/hip_runtime.h>

#include <string>

#include "../../include/cas.h"

namespace cas {

// Records msg as this thread's last error and returns s.
cas_status_t set_error(cas_status_t s, const std::string &msg);
// CAS_ERR_HIP with the HIP error's text.
cas_status_t set_hip_error(const char *what, hipError_t e);

// One host <-> device copy of a list; bytes == 0 entries are skipped.
struct HostCopy {
  const void *src;
  void *dst;
  size_t bytes;
};
// Enqueues the copies on stream s in list order. Runs of consecutive entries
// that continue both the previous source and the previous destination go out
// as one transfer (fewer, larger DMA transfers keep the host link busier).
hipError_t enqueue_copies(const HostCopy *c, int n, hipMemcpyKind kind, hipStream_t s);

}  // namespace cas
