// Host runtime of libapack: thread-local errors, version, helper counts and
// the pinned staging pool.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "common.hpp"

namespace apack {

static thread_local std::string g_error;

apack_status fail(apack_status s, const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return s;
}

void clear_error() { g_error.clear(); }

apack_status launch_status(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(APACK_E_HIP, "launch of %s failed: %s", what, hipGetErrorString(e));
  return APACK_OK;
}

// ---------------------------------------------------------------------------
// Pinned staging pool.  Blocks are reused once the event recorded after their
// last upload has completed; a busy pool grows instead of waiting, up to
// kMaxStaging blocks per device.  Past that, a call waits for the upload of
// the oldest block that is large enough and takes it, so a caller that queues
// many calls ahead holds at most that many pinned blocks.  Only when no block
// is large enough is the oldest one freed and allocated again: freeing pinned
// memory waits for the device, which would drain the caller's queue.  Blocks
// are at least kMinStaging bytes, so calls of different sizes share them.
// ---------------------------------------------------------------------------
constexpr int kMaxStaging = 32;
constexpr size_t kMinStaging = size_t(1) << 18;
struct Staging {
  void* host = nullptr;
  void* mapped = nullptr;  // device address of `host`
  size_t cap = 0;
  int device = -1;
  hipEvent_t done = nullptr;
  bool busy = false;
  uint64_t stamp = 0;      // acquisition order, for the wait at the cap
};

static std::mutex g_pool_mu;
static std::vector<Staging*> g_pool;
static uint64_t g_stamp = 0;

// Pinned memory of `cap` bytes, its device address, and the block's event
// (created once per block).
static apack_status staging_alloc(Staging* s, size_t cap) {
  s->cap = cap;
  hipError_t e = hipHostMalloc(&s->host, s->cap, hipHostMallocDefault);
  if (e != hipSuccess) {
    s->host = nullptr;
    s->cap = 0;
    return fail(APACK_E_HIP, "hipHostMalloc(%zu): %s", cap, hipGetErrorString(e));
  }
  e = hipHostGetDevicePointer(&s->mapped, s->host, 0);
  // The event only tells the host that the upload kernel has finished reading
  // the block; no device write has to become visible to the host, so it skips
  // the system-scope release (an L2 writeback that stalled the stream ~5 us).
  if (e == hipSuccess && !s->done)
    e = hipEventCreateWithFlags(&s->done, hipEventDisableTiming | hipEventDisableSystemFence);
  if (e != hipSuccess) {
    (void)hipHostFree(s->host);
    s->host = nullptr;
    s->cap = 0;
    return fail(APACK_E_HIP, "staging block set-up: %s", hipGetErrorString(e));
  }
  return APACK_OK;
}

apack_status staging_acquire(size_t bytes, Staging** blk, void** host) {
  int dev = 0;
  APACK_HIP(hipGetDevice(&dev));
  const size_t want = align_up(bytes < kMinStaging ? kMinStaging : bytes, 65536);
  std::lock_guard<std::mutex> lk(g_pool_mu);
  int on_dev = 0;
  Staging* oldest = nullptr;      // oldest block on this device
  Staging* oldest_fit = nullptr;  // oldest block large enough for this call
  for (Staging* s : g_pool) {
    if (s->device != dev) continue;
    ++on_dev;
    if (!oldest || s->stamp < oldest->stamp) oldest = s;
    if (s->cap < bytes) continue;
    if (!oldest_fit || s->stamp < oldest_fit->stamp) oldest_fit = s;
    if (s->busy) {
      hipError_t q = hipEventQuery(s->done);
      if (q == hipErrorNotReady) continue;
      if (q != hipSuccess) return fail(APACK_E_HIP, "hipEventQuery: %s", hipGetErrorString(q));
      s->busy = false;
    }
    s->busy = true;
    s->stamp = ++g_stamp;
    *blk = s;
    *host = s->host;
    return APACK_OK;
  }
  if (on_dev >= kMaxStaging) {
    // At the cap: wait until the upload of the oldest block that fits has
    // been read and reuse it; reallocate the oldest block only if none fits.
    Staging* s = oldest_fit ? oldest_fit : oldest;
    if (s->busy) APACK_HIP(hipEventSynchronize(s->done));
    s->busy = false;
    if (s->cap < bytes) {
      APACK_HIP(hipHostFree(s->host));
      s->host = nullptr;
      s->cap = 0;
      apack_status st = staging_alloc(s, want);
      if (st != APACK_OK) return st;   // the block stays idle, with no memory, until re-sized
    }
    s->busy = true;
    s->stamp = ++g_stamp;
    *blk = s;
    *host = s->host;
    return APACK_OK;
  }
  auto* s = new Staging();
  s->device = dev;
  apack_status st = staging_alloc(s, want);
  if (st != APACK_OK) {
    if (s->done) (void)hipEventDestroy(s->done);
    delete s;
    return st;
  }
  s->busy = true;
  s->stamp = ++g_stamp;
  g_pool.push_back(s);
  *blk = s;
  *host = s->host;
  return APACK_OK;
}

// The upload is a kernel that reads the mapped pinned block over PCIe: it
// stays on the caller's queue, so no copy-engine hand-off sits between the
// previous kernel and the next.
__global__ __launch_bounds__(256) void k_upload(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

apack_status staging_upload(Staging* blk, void* dst, size_t bytes, hipStream_t stream) {
  hipError_t e = hipSuccess;
  if (bytes % 16 == 0 && ((uintptr_t)dst % 16) == 0) {
    const int64_t n = (int64_t)(bytes / 16);
    const unsigned grid = (unsigned)std::min<int64_t>((n + 255) / 256, 256);
    if (n > 0) {
      hipLaunchKernelGGL(k_upload, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(blk->mapped),
                         static_cast<uint4*>(dst), n);
      e = hipGetLastError();
    }
  } else {
    e = hipMemcpyAsync(dst, blk->host, bytes, hipMemcpyHostToDevice, stream);
  }
  if (e != hipSuccess) {
    std::lock_guard<std::mutex> lk(g_pool_mu);
    blk->busy = false;  // nothing was enqueued that still reads the block
    return fail(APACK_E_HIP, "staging upload: %s", hipGetErrorString(e));
  }
  return APACK_OK;
}

apack_status staging_release(Staging* blk, hipStream_t stream) {
  // If the record fails the block stays busy for good: the upload may still
  // be queued, so it cannot be handed out again.
  const hipError_t e = hipEventRecord(blk->done, stream);
  if (e != hipSuccess) return fail(APACK_E_HIP, "staging event: %s", hipGetErrorString(e));
  return APACK_OK;
}

}  // namespace apack

using namespace apack;

extern "C" {

const char* apack_version(void) { return "apack 0.1 (gfx950)"; }

const char* apack_last_error(void) { return g_error.c_str(); }

const char* apack_status_string(apack_status s) {
  switch (s) {
    case APACK_OK: return "ok";
    case APACK_E_ARG: return "bad argument";
    case APACK_E_SHAPE: return "inconsistent shapes";
    case APACK_E_DTYPE: return "bad dtype";
    case APACK_E_WORKSPACE: return "workspace too small or misaligned";
    case APACK_E_ALIAS: return "output overlaps input";
    case APACK_E_HIP: return "HIP runtime error";
    case APACK_E_UNSUPPORTED: return "unsupported configuration";
  }
  return "unknown status";
}

int64_t apack_keep_count(double keep, int64_t n) {
  if (!(keep >= 0.0 && keep <= 1.0) || n < 0) return -1;
  const double x = keep * static_cast<double>(n);
  const double slack = std::ldexp(static_cast<double>(n), -50);
  int64_t k = static_cast<int64_t>(std::ceil(x - slack));
  if (k < 0) k = 0;
  if (k > n) k = n;
  return k;
}

int64_t apack_visual_budget(double r_pre, int64_t n_audio, int64_t n_visual) {
  if (n_audio < 0 || n_visual < 0) return -1;
  int64_t b = apack_keep_count(r_pre, n_audio + n_visual);
  if (b < 0) return -1;
  b -= n_audio;
  if (b < 0) b = 0;
  if (b > n_visual) b = n_visual;
  return b;
}

void apack_dyn_params_default(apack_dyn_params* p) {
  if (!p) return;
  p->window = 3;
  p->dafps_k = 5;
  p->tau_gate = 0.78;
  p->beta = 0.90;
  p->gamma = 0.9;
  p->tau_sim = 0.97;
  p->sigma = 1.0;
  p->lambda_seg = 0.5;
  p->cover_thresh = 0.8;
  p->dafps_power = 0.5;
  p->r_pre = 0.50;
  p->alignment = APACK_ALIGN_GATED_CKA;
}

}  // extern "C"
