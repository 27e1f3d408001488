// In-place stable compaction of the kept rows (Section 3.2: the pruned
// tokens' key and value entries are removed; Algorithm 1: slice their
// KV-cache entries), for callers that cannot hold the cache twice.
//
// For every plane x (each K/V head plane, the hidden states, each position
// row):  x[i] = x[src[i]] for i < n_out, with src strictly increasing, so
// src[i] >= i and a row only ever moves towards the front.  The hazard is a
// store into row r that lands before an earlier output row j (src[j] = r,
// j < r) has read row r.
//
// Output rows are cut into stripes of kStripe rows.  The readers of the rows
// of stripe s are output rows j <= r, so they sit in stripes <= s, and since
// src is increasing they form one run [first_reader[s], first_reader[s+1]).
// Work items are (stripe, slice of one plane) in stripe-major order and are
// claimed through a ticket counter in that order, kGroup items at a time.
// An item loads its source rows into registers, counts itself as read in its
// stripe's counter, waits until every earlier stripe holding readers of its
// destination rows has been read completely, then stores.  Readers inside the
// item's own stripe and plane are the item itself: a workgroup barrier
// separates its loads from its stores.
//
// Why it drains: an item counts itself as read before it waits, and it only
// waits on strictly earlier stripes, whose items hold smaller tickets and so
// were claimed by running workgroups.  By induction over stripes every
// counter fills.  This holds for any src; only the row contents need src to
// be strictly increasing.
//
// Each wait is still bounded (a defensive limit of ~seconds of polling, see
// apack_set_inplace_wait_limit).  A wait that gives up sets the error word
// in the workspace and its ticket stores nothing, so no source row that an
// earlier stripe has yet to read is ever overwritten; the caller learns of
// it from apack_compact_kv_inplace_status.
#include <algorithm>
#include <array>
#include <atomic>
#include <cstring>
#include <mutex>

#include "common.hpp"
#include "sync.hpp"

namespace apack {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxTensors = 128;           // 64 layers x {K, V}
constexpr int kThreads = 512;
constexpr int kPerThread = 4;
constexpr int kSlice = 16;                 // units per row slice (256 bytes at 16-byte units)
constexpr int kStripe = kThreads * kPerThread / kSlice;  // output rows per stripe
constexpr int kGroup = 2;                  // items per ticket, loaded together
constexpr int kCounterPad = 16;            // one 64-byte line per stripe counter
constexpr int kMaxPosRows = kThreads * kPerThread / kStripe;
constexpr uint32_t kDefaultWaitLimit = 1u << 22;  // polls per wait (~seconds)

struct InplaceArgs {
  const int32_t* src;
  int64_t n_out, n_in;
  int64_t n_stripes, n_items;
  int32_t items_per_stripe;
  uint32_t wait_limit;     // polls before a wait gives up; 0: every wait gives up at once
  // K/V planes: tensor t, head h at planes[t] + h * hs; rows of kv_row_units.
  int32_t kv_planes, heads, kv_slices;
  int64_t kv_row_units, hs;
  // Hidden states [rows][h_row_units units], cut into h_slices slices.
  void* hid;
  int32_t h_slices;
  int64_t h_row_units;
  // Position ids [p_rows][p_stride] int32 (one item per stripe).
  int32_t* pos;
  int32_t p_rows;
  int64_t p_stride;
  // Workspace.
  uint32_t* ticket;
  uint32_t* err;
  uint32_t* done;          // [n_stripes][kCounterPad]
  const int32_t* first_reader;  // [n_stripes + 1]
  void* planes[kMaxTensors];
};

__device__ __forceinline__ int64_t floor_div(int64_t a, int64_t b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

// Zeroes the ticket and the stripe counters and fills first_reader[s], the
// first output row j with src[j] >= s * kStripe (n_out when there is none).
__global__ __launch_bounds__(kThreads) void k_inplace_prep(const InplaceArgs a) {
  const int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  int32_t* fr = const_cast<int32_t*>(a.first_reader);
  if (g == 0) {
    *a.ticket = 0u;
    *a.err = 0u;
  }
  if (g < a.n_stripes) a.done[g * kCounterPad] = 0u;
  if (g >= a.n_out) return;
  const int64_t prev = g == 0 ? -1 : (int64_t)a.src[g - 1];
  const int64_t cur = a.src[g];
  // Stripes s with src[g-1] < s * kStripe <= src[g] take g.
  const int64_t lo = std::max<int64_t>(floor_div(prev, kStripe) + 1, 0);
  const int64_t hi = std::min<int64_t>(floor_div(cur, kStripe), a.n_stripes);
  for (int64_t s = lo; s <= hi; ++s) fr[s] = (int32_t)g;
  if (g == a.n_out - 1)
    for (int64_t s = std::max<int64_t>(floor_div(cur, kStripe) + 1, 0); s <= a.n_stripes; ++s) fr[s] = (int32_t)a.n_out;
}

// Blocks until every stripe in [lo, hi] has all of its items read; false
// (with the workspace's error word set) if a wait gave up first.  A limit
// of 0 gives up on any non-empty range without polling.
__device__ bool wait_stripes(const InplaceArgs& a, int64_t lo, int64_t hi) {
  if (a.wait_limit == 0 && lo <= hi) {
    __hip_atomic_fetch_or(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return false;
  }
  for (int64_t st = lo; st <= hi; ++st) {
    const uint32_t* c = a.done + st * kCounterPad;
    uint32_t spins = 0;
    while (ld_agent(c) < (uint32_t)a.items_per_stripe) {
      if (++spins > a.wait_limit) {
        __hip_atomic_fetch_or(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return false;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  return true;
}

// Position ids move as 4-byte words inside a unit of either width.
__device__ __forceinline__ void put_word(uint32_t& u, uint32_t x) { u = x; }
__device__ __forceinline__ void put_word(u32x4& u, uint32_t x) { u.x = x; }
__device__ __forceinline__ uint32_t get_word(uint32_t u) { return u; }
__device__ __forceinline__ uint32_t get_word(const u32x4& u) { return u.x; }

// One item's share of one thread: up to kPerThread units loaded from the
// source rows, with a bit per unit that has somewhere to go.
template <class U>
struct ItemRegs {
  U v[kPerThread];
  uint32_t live;
};

// Geometry of item k of a stripe: base, row stride and slice of a K/V plane
// or of the hidden states (units of U); positions use their own path.
template <class U>
struct Slice {
  U* base;
  int64_t stride;
  int c0, w;
  bool pos;
};

template <class U>
__device__ __forceinline__ Slice<U> slice_of(const InplaceArgs& a, int k) {
  Slice<U> g{nullptr, 0, 0, 0, false};
  const int kv_items = a.kv_planes * a.kv_slices;
  if (k < kv_items) {
    const int plane = k / a.kv_slices, sl = k % a.kv_slices;
    g.base = static_cast<U*>(a.planes[plane / a.heads]) + (plane % a.heads) * a.hs;
    g.stride = a.kv_row_units;
    g.c0 = sl * kSlice;
    g.w = (int)std::min<int64_t>(kSlice, a.kv_row_units - g.c0);
  } else if (k < kv_items + a.h_slices) {
    g.base = static_cast<U*>(a.hid);
    g.stride = a.h_row_units;
    g.c0 = (k - kv_items) * kSlice;
    g.w = (int)std::min<int64_t>(kSlice, a.h_row_units - g.c0);
  } else {
    g.pos = true;
  }
  return g;
}

// Unit i of this thread in an item of stripe s: destination row r and
// column c (position items: position row c), or false if there is none.
template <class U>
__device__ __forceinline__ bool unit_of(const InplaceArgs& a, const Slice<U>& g, int64_t s, int i, int64_t& r,
                                        int& c) {
  const int u = threadIdx.x + i * kThreads;
  if (!g.pos) {
    r = s * kStripe + u / kSlice;
    c = u % kSlice;
    return c < g.w && r < a.n_out;
  }
  r = s * kStripe + u % kStripe;
  c = u / kStripe;
  return c < a.p_rows && r < a.n_out;
}

// sidx holds src of the rows of stripes sa, sa + 1, ... (kStripe each).
template <class U>
__device__ __forceinline__ void load_item(const InplaceArgs& a, int64_t item, const int32_t* sidx, int64_t sa,
                                          ItemRegs<U>& q) {
  const int64_t s = item / a.items_per_stripe;
  const Slice<U> g = slice_of<U>(a, (int)(item % a.items_per_stripe));
  q.live = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    int64_t r;
    int c;
    if (!unit_of(a, g, s, i, r, c)) continue;
    const int64_t sr = sidx[(s - sa) * kStripe + (r - s * kStripe)];
    if (sr < 0 || sr >= a.n_in || sr == r) continue;   // nothing to move
    if (!g.pos) {
      q.v[i] = __builtin_nontemporal_load(g.base + sr * g.stride + g.c0 + c);
    } else {
      put_word(q.v[i], __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(a.pos) + c * a.p_stride + sr));
    }
    q.live |= 1u << i;
  }
}

template <class U>
__device__ __forceinline__ void store_item(const InplaceArgs& a, int64_t item, const ItemRegs<U>& q) {
  const int64_t s = item / a.items_per_stripe;
  const Slice<U> g = slice_of<U>(a, (int)(item % a.items_per_stripe));
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    if (!(q.live >> i & 1u)) continue;
    int64_t r;
    int c;
    unit_of(a, g, s, i, r, c);
    if (!g.pos)
      __builtin_nontemporal_store(q.v[i], g.base + r * g.stride + g.c0 + c);
    else
      __builtin_nontemporal_store(get_word(q.v[i]), reinterpret_cast<uint32_t*>(a.pos) + c * a.p_stride + r);
  }
}

// Stripes in [lo, hi] whose items are not all read yet: true if any.
__device__ __forceinline__ bool stripes_pending(const InplaceArgs& a, int64_t lo, int64_t hi) {
  bool pending = false;
  for (int64_t st = lo; st <= hi; ++st) pending |= ld_agent(a.done + st * kCounterPad) < (uint32_t)a.items_per_stripe;
  return pending;
}

// Earlier stripes holding readers of the rows of stripe t, as [lo, hi]
// (empty when lo > hi), from first_reader[t] and first_reader[t + 1].
__device__ __forceinline__ void reader_stripes(const InplaceArgs& a, int64_t t, int32_t f0, int32_t f1, int64_t& lo,
                                               int64_t& hi) {
  const int64_t j0 = std::clamp<int64_t>(f0, 0, a.n_out);
  const int64_t j1 = std::clamp<int64_t>(f1, j0, a.n_out);
  lo = j0 / kStripe;
  hi = j1 > j0 ? std::min<int64_t>((j1 - 1) / kStripe, t - 1) : -1;
}

// A workgroup claims kGroup items with one ticket, loads them all, counts
// them read in their stripes' counters, then waits for the readers of their
// destination rows, then stores (nothing, if a wait gave up), and only then
// claims its next ticket.  So
// a workgroup never waits while it holds a claimed item it has not counted:
// a count waits on nothing but its own loads, and no chain of waits forms
// between stripes.  Thread 0 reads the reader ranges before the data loads
// and looks at the counters once while those loads are in flight; it blocks
// after counting only if some reader stripe was incomplete then.
template <class U>
__global__ __launch_bounds__(kThreads) void k_compact_inplace(const InplaceArgs a) {
  __shared__ uint32_t sh_ticket;
  __shared__ uint32_t sh_ok;                   // the ticket's waits all completed
  __shared__ int32_t sidx[kGroup * kStripe];   // src of the ticket's output rows
  const int tid = threadIdx.x;
  int64_t waited = -1;  // latest stripe whose readers thread 0 has seen complete
  for (;;) {
    if (tid == 0) sh_ticket = __hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int64_t i0 = (int64_t)sh_ticket * kGroup;
    if (i0 >= a.n_items) break;
    const int64_t i1 = std::min<int64_t>(i0 + kGroup, a.n_items);
    const int64_t sb = (i1 - 1) / a.items_per_stripe;
    // Thread 0: reader ranges of the ticket's stripes not yet seen complete.
    int32_t fr[kGroup + 1];
    const int64_t t0 = std::max(waited + 1, i0 / a.items_per_stripe);
    if (tid == 0)
#pragma unroll
      for (int j = 0; j <= kGroup; ++j) fr[j] = t0 + j <= sb + 1 ? a.first_reader[t0 + j] : 0;
    // The ticket's items lie in at most kGroup stripes; their source rows
    // are read once into LDS (one index load per row, not one per unit).
    // The previous ticket's reads of sidx ended before its count barrier.
    const int64_t sa = i0 / a.items_per_stripe;
    for (int j = tid; j < (int)(sb - sa + 1) * kStripe; j += kThreads) {
      const int64_t r = sa * kStripe + j;
      sidx[j] = r < a.n_out ? a.src[r] : -1;
    }
    __syncthreads();
    ItemRegs<U> q[kGroup];
#pragma unroll
    for (int p = 0; p < kGroup; ++p) {
      q[p].live = 0;
      if (i0 + p < i1) load_item<U>(a, i0 + p, sidx, sa, q[p]);
    }
    bool pending = false;
    if (tid == 0)
#pragma unroll
      for (int j = 0; j < kGroup; ++j)
        if (t0 + j <= sb) {
          int64_t lo, hi;
          reader_stripes(a, t0 + j, fr[j], fr[j + 1], lo, hi);
          pending |= stripes_pending(a, lo, hi);
        }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
      for (int64_t i = i0; i < i1; ++i)
        __hip_atomic_fetch_add(a.done + i / a.items_per_stripe * kCounterPad, 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
      bool ok = true;
      if (pending || a.wait_limit == 0)
        for (int j = 0; j < kGroup; ++j)
          if (t0 + j <= sb) {
            int64_t lo, hi;
            reader_stripes(a, t0 + j, fr[j], fr[j + 1], lo, hi);
            ok = ok && wait_stripes(a, lo, hi);
          }
      if (ok) waited = std::max(waited, sb);
      sh_ok = ok ? 1u : 0u;
    }
    __syncthreads();
    if (sh_ok) {
#pragma unroll
      for (int p = 0; p < kGroup; ++p)
        if (q[p].live) store_item<U>(a, i0 + p, q[p]);
    }
  }
}

struct InplaceLayout {
  size_t off_ticket, off_done, off_fr, bytes;
};

InplaceLayout inplace_layout(int64_t n_out) {
  const int64_t n_stripes = (n_out + kStripe - 1) / kStripe;
  Carver c(nullptr);
  InplaceLayout l;
  l.off_ticket = c.used;
  c.take<uint32_t>(2);
  l.off_done = c.used;
  c.take<uint32_t>((size_t)n_stripes * kCounterPad);
  l.off_fr = c.used;
  c.take<int32_t>((size_t)n_stripes + 1);
  l.bytes = c.used;
  return l;
}

int resident_groups() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_compact_inplace<u32x4>, kThreads, 0) != hipSuccess ||
        per_cu <= 0)
      per_cu = 4;
    n = std::max(1, cus * per_cu);
  }
  return n;
}

std::atomic<uint32_t> g_wait_limit{kDefaultWaitLimit};

}  // namespace

// Library-owned scratch of apack_compact_kv_inplace_static: the workspace of
// a compaction of up to kStaticRows kept rows (ticket, status word, one
// counter line per stripe and the stripes' first readers), one copy per
// GPU, held until the process ends.  Host code never uses this name as an
// address: each device's copy is reached through the pointer that
// hipGetSymbolAddress returns on that device.
constexpr int64_t kStaticRows = int64_t(1) << 20;
constexpr int64_t kStaticStripes = kStaticRows / kStripe;
constexpr size_t kStaticBytes = 256 + (size_t)kStaticStripes * kCounterPad * 4 +
                                ((size_t)(kStaticStripes + 1) * 4 + 255) / 256 * 256;
static __device__ __align__(256) uint8_t scratch[kStaticBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
std::array<void*, kMaxDevices> g_scratch{};   // device address of scratch, per device

// The address of the current device's copy of `scratch`, looked up once per
// device with that device current.
apack_status static_scratch(void** ptr) {
  int dev = 0;
  APACK_HIP(hipGetDevice(&dev));
  APACK_CHECK(dev >= 0 && dev < kMaxDevices, APACK_E_UNSUPPORTED, "device %d beyond the %d the library tracks", dev,
              kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    APACK_CHECK(e == hipSuccess && p, APACK_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return APACK_OK;
}

apack_status compact_inplace(int64_t n_out, const int32_t* src_rows, int64_t n_in, int32_t n_layers,
                             void* const* k, void* const* v, int32_t hkv, int32_t d, apack_dtype dtype,
                             int64_t head_stride, void* hidden, int32_t hidden_dim, int32_t* pos, int32_t pos_rows,
                             int64_t pos_stride, void* workspace, size_t workspace_bytes, void* stream);

}  // namespace
}  // namespace apack

using namespace apack;

extern "C" size_t apack_compact_kv_inplace_workspace(int64_t n_out) {
  return n_out < 0 ? 0 : inplace_layout(n_out).bytes;
}

extern "C" uint32_t apack_set_inplace_wait_limit(uint32_t polls) { return g_wait_limit.exchange(polls); }

extern "C" apack_status apack_compact_kv_inplace_status(const void* workspace, size_t workspace_bytes,
                                                        int32_t* gave_up, void* stream) {
  clear_error();
  APACK_CHECK(gave_up, APACK_E_ARG, "gave_up is NULL");
  APACK_CHECK(workspace && ((uintptr_t)workspace % kAlign) == 0, APACK_E_WORKSPACE,
              "workspace must be non-NULL and %zu-byte aligned", kAlign);
  const InplaceLayout lay = inplace_layout(0);
  APACK_CHECK(workspace_bytes >= lay.off_ticket + 2 * sizeof(uint32_t), APACK_E_WORKSPACE,
              "workspace of %zu bytes holds no status word", workspace_bytes);
  uint32_t err = 0;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  APACK_HIP(hipMemcpyAsync(&err, static_cast<const char*>(workspace) + lay.off_ticket + sizeof(uint32_t),
                           sizeof err, hipMemcpyDeviceToHost, hs));
  APACK_HIP(hipStreamSynchronize(hs));
  *gave_up = err != 0 ? 1 : 0;
  return APACK_OK;
}

extern "C" apack_status apack_compact_kv_inplace(int64_t n_out, const int32_t* src_rows, int64_t n_in,
                                                 int32_t n_layers, void* const* k, void* const* v, int32_t hkv,
                                                 int32_t d, apack_dtype dtype, int64_t head_stride, void* hidden,
                                                 int32_t hidden_dim, int32_t* pos, int32_t pos_rows,
                                                 int64_t pos_stride, void* workspace, size_t workspace_bytes,
                                                 void* stream) {
  clear_error();
  return compact_inplace(n_out, src_rows, n_in, n_layers, k, v, hkv, d, dtype, head_stride, hidden, hidden_dim, pos,
                         pos_rows, pos_stride, workspace, workspace_bytes, stream);
}

extern "C" apack_status apack_compact_kv_inplace_static(int64_t n_out, const int32_t* src_rows, int64_t n_in,
                                                        int32_t n_layers, void* const* k, void* const* v,
                                                        int32_t hkv, int32_t d, apack_dtype dtype,
                                                        int64_t head_stride, void* hidden, int32_t hidden_dim,
                                                        int32_t* pos, int32_t pos_rows, int64_t pos_stride,
                                                        void* stream) {
  clear_error();
  APACK_CHECK(n_out <= kStaticRows, APACK_E_UNSUPPORTED,
              "n_out (%lld) exceeds the %lld kept rows the static scratch holds", (long long)n_out,
              (long long)kStaticRows);
  void* ws = nullptr;
  if (n_out > 0) {
    const apack_status st = static_scratch(&ws);
    if (st != APACK_OK) return st;
  }
  return compact_inplace(n_out, src_rows, n_in, n_layers, k, v, hkv, d, dtype, head_stride, hidden, hidden_dim, pos,
                         pos_rows, pos_stride, ws, kStaticBytes, stream);
}

namespace apack {
namespace {

// Validation and launch of one in-place compaction (both entry points).
apack_status compact_inplace(int64_t n_out, const int32_t* src_rows, int64_t n_in, int32_t n_layers,
                             void* const* k, void* const* v, int32_t hkv, int32_t d, apack_dtype dtype,
                             int64_t head_stride, void* hidden, int32_t hidden_dim, int32_t* pos, int32_t pos_rows,
                             int64_t pos_stride, void* workspace, size_t workspace_bytes, void* stream) {
  APACK_CHECK(dtype_ok(dtype), APACK_E_DTYPE, "unknown dtype %d", (int)dtype);
  APACK_CHECK(n_out >= 0 && n_in >= 0, APACK_E_SHAPE, "negative row count");
  APACK_CHECK(n_out <= n_in, APACK_E_SHAPE, "n_out (%lld) exceeds n_in (%lld)", (long long)n_out,
              (long long)n_in);
  APACK_CHECK(n_in < (int64_t(1) << 31), APACK_E_UNSUPPORTED, "row counts must be < 2^31");
  APACK_CHECK(n_layers >= 0 && n_layers <= kMaxTensors / 2, APACK_E_ARG, "n_layers must lie in [0, %d]",
              kMaxTensors / 2);
  APACK_CHECK(hidden_dim >= 0 && pos_rows >= 0, APACK_E_ARG, "negative hidden_dim or pos_rows");
  APACK_CHECK(pos_rows <= kMaxPosRows, APACK_E_UNSUPPORTED, "at most %d position rows", kMaxPosRows);
  APACK_CHECK(n_out == 0 || src_rows, APACK_E_ARG, "src_rows is NULL");
  const size_t es = dtype_size(dtype);
  const bool has_v = v != nullptr;
  if (n_layers > 0) {
    APACK_CHECK(k != nullptr, APACK_E_ARG, "K pointer table must be non-NULL");
    APACK_CHECK(hkv > 0 && d > 0, APACK_E_SHAPE, "hkv and d must be positive");
    APACK_CHECK(head_stride >= n_in * d, APACK_E_SHAPE, "head stride must be >= rows * d");
  }
  const bool has_h = hidden_dim > 0;
  const bool has_p = pos_rows > 0;
  if (has_h) APACK_CHECK(hidden, APACK_E_ARG, "hidden must be non-NULL");
  if (has_p) {
    APACK_CHECK(pos, APACK_E_ARG, "pos must be non-NULL");
    APACK_CHECK(pos_stride >= n_in, APACK_E_SHAPE, "position row stride must be >= rows");
  }
  // Every plane is distinct; src_rows and the workspace touch none of them.
  // (A fixed table: this path allocates nothing, on the host or the device.)
  struct Buf {
    const void* p;
    size_t bytes;
  };
  Buf bufs[kMaxTensors + 2];
  int n_bufs = 0;
  const size_t kv_bytes = n_layers ? (size_t)((hkv - 1) * head_stride + n_in * d) * es : 0;
  for (int l = 0; l < n_layers; ++l) {
    APACK_CHECK(k[l] && (!has_v || v[l]), APACK_E_ARG, "layer %d: NULL K/V pointer", l);
    bufs[n_bufs++] = Buf{k[l], kv_bytes};
    if (has_v) bufs[n_bufs++] = Buf{v[l], kv_bytes};
  }
  if (has_h) bufs[n_bufs++] = Buf{hidden, (size_t)n_in * hidden_dim * es};
  if (has_p) bufs[n_bufs++] = Buf{pos, (size_t)((pos_rows - 1) * pos_stride + n_in) * 4};
  for (int i = 0; i < n_bufs; ++i)
    for (int j = i + 1; j < n_bufs; ++j)
      APACK_CHECK(!overlaps(bufs[i].p, bufs[i].bytes, bufs[j].p, bufs[j].bytes), APACK_E_ALIAS,
                  "two compacted tensors overlap");
  const InplaceLayout lay = inplace_layout(n_out);
  if (n_out > 0) {
    APACK_CHECK(workspace && ((uintptr_t)workspace % kAlign) == 0, APACK_E_WORKSPACE,
                "workspace must be non-NULL and %zu-byte aligned", kAlign);
    APACK_CHECK(workspace_bytes >= lay.bytes, APACK_E_WORKSPACE, "workspace of %zu bytes < %zu needed",
                workspace_bytes, lay.bytes);
    for (int i = 0; i < n_bufs; ++i) {
      APACK_CHECK(!overlaps(bufs[i].p, bufs[i].bytes, src_rows, (size_t)n_out * 4), APACK_E_ALIAS,
                  "src_rows overlaps a compacted tensor");
      APACK_CHECK(!overlaps(bufs[i].p, bufs[i].bytes, workspace, lay.bytes), APACK_E_ALIAS,
                  "the workspace overlaps a compacted tensor");
    }
    APACK_CHECK(!overlaps(src_rows, (size_t)n_out * 4, workspace, lay.bytes), APACK_E_ALIAS,
                "the workspace overlaps src_rows");
  }
  if (n_out == 0) return APACK_OK;

  // 16-byte units when every row, stride and base allows it, else 4 bytes.
  const int64_t kv_row_bytes = (int64_t)d * (int64_t)es;
  auto al = [](const void* p, uintptr_t b) { return ((uintptr_t)p % b) == 0; };
  bool wide = true;
  if (n_layers) {
    wide &= kv_row_bytes % 16 == 0 && (head_stride * (int64_t)es) % 16 == 0;
    for (int l = 0; l < n_layers; ++l) wide &= al(k[l], 16) && (!has_v || al(v[l], 16));
  }
  if (has_h) wide &= ((int64_t)hidden_dim * (int64_t)es) % 16 == 0 && al(hidden, 16);
  if (!wide) {
    APACK_CHECK(kv_row_bytes % 4 == 0 && ((int64_t)hidden_dim * (int64_t)es) % 4 == 0, APACK_E_UNSUPPORTED,
                "row sizes must be multiples of 4 bytes");
    for (int l = 0; l < n_layers; ++l)
      APACK_CHECK(al(k[l], 4) && (!has_v || al(v[l], 4)), APACK_E_ARG, "K/V pointers must be 4-byte aligned");
    if (has_h) APACK_CHECK(al(hidden, 4), APACK_E_ARG, "hidden must be 4-byte aligned");
  }
  if (has_p) APACK_CHECK(al(pos, 4), APACK_E_ARG, "pos must be 4-byte aligned");
  const int64_t ub = wide ? 16 : 4;

  InplaceArgs a;
  std::memset(&a, 0, sizeof a);
  a.src = src_rows;
  a.n_out = n_out;
  a.n_in = n_in;
  a.n_stripes = (n_out + kStripe - 1) / kStripe;
  a.heads = n_layers ? hkv : 1;
  if (n_layers) {
    const int n_tensors = (has_v ? 2 : 1) * n_layers;
    a.kv_planes = n_tensors * hkv;
    a.kv_row_units = kv_row_bytes / ub;
    a.kv_slices = (int32_t)((a.kv_row_units + kSlice - 1) / kSlice);
    a.hs = head_stride * (int64_t)es / ub;
    for (int l = 0; l < n_layers; ++l) {
      if (has_v) {
        a.planes[2 * l] = k[l];
        a.planes[2 * l + 1] = v[l];
      } else {
        a.planes[l] = k[l];
      }
    }
  }
  if (has_h) {
    a.hid = hidden;
    a.h_row_units = (int64_t)hidden_dim * (int64_t)es / ub;
    a.h_slices = (int32_t)((a.h_row_units + kSlice - 1) / kSlice);
  }
  if (has_p) {
    a.pos = pos;
    a.p_rows = pos_rows;
    a.p_stride = pos_stride;
  }
  const int64_t ips = (int64_t)a.kv_planes * a.kv_slices + a.h_slices + (has_p ? 1 : 0);
  if (ips == 0) return APACK_OK;
  APACK_CHECK(ips * a.n_stripes < (int64_t(1) << 31) * kGroup, APACK_E_UNSUPPORTED, "too many work items");
  a.items_per_stripe = (int32_t)ips;
  a.n_items = ips * a.n_stripes;
  a.wait_limit = g_wait_limit.load();
  char* ws = static_cast<char*>(workspace);
  a.ticket = reinterpret_cast<uint32_t*>(ws + lay.off_ticket);
  a.err = a.ticket + 1;
  a.done = reinterpret_cast<uint32_t*>(ws + lay.off_done);
  a.first_reader = reinterpret_cast<const int32_t*>(ws + lay.off_fr);

  hipStream_t hs = static_cast<hipStream_t>(stream);
  const int64_t prep_threads = std::max<int64_t>(n_out, a.n_stripes + 1);
  hipLaunchKernelGGL(k_inplace_prep, dim3((unsigned)((prep_threads + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     hs, a);
  apack_status st = launch_status("k_inplace_prep");
  if (st != APACK_OK) return st;
  const int64_t tickets = (a.n_items + kGroup - 1) / kGroup;
  const unsigned grid = (unsigned)std::min<int64_t>(tickets, resident_groups());
  if (wide)
    hipLaunchKernelGGL(k_compact_inplace<u32x4>, dim3(grid), dim3(kThreads), 0, hs, a);
  else
    hipLaunchKernelGGL(k_compact_inplace<uint32_t>, dim3(grid), dim3(kThreads), 0, hs, a);
  return launch_status("k_compact_inplace");
}

}  // namespace
}  // namespace apack
