// Shared host-side runtime of libapack: error reporting, checked HIP calls,
// workspace carving and the pinned staging pool that carries host
// descriptors to the device without synchronising.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <string>

#include "apack.h"

namespace apack {

// Sets the thread-local error message and returns `s`.
apack_status fail(apack_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

#define APACK_HIP(expr)                                                              \
  do {                                                                               \
    hipError_t e_ = (expr);                                                          \
    if (e_ != hipSuccess)                                                            \
      return ::apack::fail(APACK_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define APACK_CHECK(cond, status, ...)                  \
  do {                                                  \
    if (!(cond)) return ::apack::fail(status, __VA_ARGS__); \
  } while (0)

// Status of the most recent kernel launch on this thread.
apack_status launch_status(const char* what);

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Carves aligned sub-buffers out of one workspace; the same code sizes the
// workspace (base == nullptr) and hands out pointers.
struct Carver {
  char* base;
  size_t used = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t count) {
    size_t off = used;
    used = align_up(used + count * sizeof(T));
    return base ? reinterpret_cast<T*>(base + off) : nullptr;
  }
};

// Pinned host staging for small descriptor uploads.  acquire() returns a
// pinned block of at least `bytes`; upload() copies it to `dst` on `stream`;
// release() (called once the call's other launches are queued, whatever their
// status) records the event that frees the block once the stream reaches it.
// Recording after the launches keeps the event's packet from sitting between
// the upload and the first kernel that reads the descriptors.
struct Staging;
apack_status staging_acquire(size_t bytes, Staging** blk, void** host);
apack_status staging_upload(Staging* blk, void* dst, size_t bytes, hipStream_t stream);
apack_status staging_release(Staging* blk, hipStream_t stream);

// Byte ranges [a, a+na) and [b, b+nb) overlap.
inline bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  auto pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return na && nb && pa < pb + nb && pb < pa + na;
}

inline size_t dtype_size(apack_dtype dt) { return dt == APACK_BF16 ? 2 : 4; }
inline bool dtype_ok(int dt) { return dt == APACK_BF16 || dt == APACK_F32; }

}  // namespace apack
