// Gather compaction of the kept rows (Section 3.2: the pruned tokens' key and
// value entries are removed; Algorithm 1: slice their KV-cache entries).
//
// One launch moves every plane: for each (tensor, head) plane of the K/V
// cache, the hidden-state rows and the position-id rows,
//   out[i] = in[src_rows[i]],  i < n_out.
// Work items are 16 KB slabs (1024 units of 16 bytes, 4 per thread) so each
// thread keeps four independent 16-byte loads in flight before its stores;
// HBM-bound by design.  The source rows of a slab are read once into LDS
// before its data loads: one index load per row rather than one per 16-byte
// unit (a 256-byte K/V row spans 16 units).  Rows whose index is outside
// [0, n_in) are skipped.
#include <algorithm>
#include <cstring>

#include "common.hpp"

namespace apack {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxTensors = 128;   // 64 layers x {K, V}
constexpr int kThreads = 256;
constexpr int kPerThread = 4;
constexpr int kItemUnits = kThreads * kPerThread;

struct GatherArgs {
  const int32_t* src;
  int64_t n_out, n_in;
  // K/V planes: tensor t, head h at base + h*head_stride.
  int32_t n_tensors, heads;
  int64_t row_units;          // units per K/V row
  int64_t hs_in, hs_out;      // head strides in units
  int64_t kv_rows_per_item, kv_items_per_plane, kv_items;
  int32_t row_magic, h_row_magic;   // div_magic(row_units), div_magic(h_row_units)
  // hidden
  const void* h_in;
  void* h_out;
  int64_t h_row_units, h_rows_per_item, h_items;
  // positions (always 4-byte units)
  const int32_t* p_in;
  int32_t* p_out;
  int32_t p_rows;
  int64_t p_stride_in, p_stride_out, p_items_per_row, p_items;
  const void* in[kMaxTensors];
  void* out[kMaxTensors];
};

// u / d for 0 <= u < 1024 and 1 <= d <= 1024 as (u * magic) >> 20 with
// magic = ceil(2^20 / d): exact on that range (the product stays below 2^30).
inline int32_t div_magic(int64_t d) { return (int32_t)(((int64_t(1) << 20) + d - 1) / d); }

// rows * row_units <= kItemUnits, so rows <= kItemUnits and row_units <= kItemUnits.
// Every thread of the workgroup calls this (it holds a barrier).  The four
// index reads from LDS are issued together, then the four data loads.
template <class U>
__device__ __forceinline__ void copy_rows(const U* __restrict__ in, U* __restrict__ out,
                                          const int32_t* __restrict__ src, int64_t r0, int rows,
                                          int row_units, int magic, int64_t n_out, int64_t n_in,
                                          int32_t* sidx) {
  for (int i = threadIdx.x; i < rows; i += kThreads) {
    const int64_t r = r0 + i;
    int32_t s = -1;
    if (r < n_out) {
      s = src[r];
      if (s < 0 || s >= n_in) s = -1;
    }
    sidx[i] = s;
  }
  __syncthreads();
  const int units = rows * row_units;
  int32_t s[kPerThread];
  int rl[kPerThread], c[kPerThread];
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int u = threadIdx.x + i * kThreads;
    rl[i] = (u * magic) >> 20;
    c[i] = u - rl[i] * row_units;
    s[i] = u < units ? sidx[rl[i]] : -1;
  }
  U v[kPerThread];
#pragma unroll
  for (int i = 0; i < kPerThread; ++i)
    if (s[i] >= 0) v[i] = __builtin_nontemporal_load(in + (int64_t)s[i] * row_units + c[i]);
#pragma unroll
  for (int i = 0; i < kPerThread; ++i)
    if (s[i] >= 0) __builtin_nontemporal_store(v[i], out + (r0 + rl[i]) * row_units + c[i]);
}

template <class U>
__global__ __launch_bounds__(kThreads) void k_gather(const GatherArgs a) {
  __shared__ int32_t sidx[kItemUnits];
  int64_t item = blockIdx.x;
  if (item < a.kv_items) {
    const int64_t plane = item / a.kv_items_per_plane;
    const int64_t r0 = (item % a.kv_items_per_plane) * a.kv_rows_per_item;
    const int t = (int)(plane / a.heads), h = (int)(plane % a.heads);
    const U* in = static_cast<const U*>(a.in[t]) + h * a.hs_in;
    U* out = static_cast<U*>(a.out[t]) + h * a.hs_out;
    copy_rows<U>(in, out, a.src, r0, (int)a.kv_rows_per_item, (int)a.row_units, a.row_magic, a.n_out, a.n_in,
                 sidx);
    return;
  }
  item -= a.kv_items;
  if (item < a.h_items) {
    copy_rows<U>(static_cast<const U*>(a.h_in), static_cast<U*>(a.h_out), a.src, item * a.h_rows_per_item,
                 (int)a.h_rows_per_item, (int)a.h_row_units, a.h_row_magic, a.n_out, a.n_in, sidx);
    return;
  }
  item -= a.h_items;
  if (item < a.p_items) {
    const int64_t row = item / a.p_items_per_row;
    const int64_t c0 = (item % a.p_items_per_row) * kItemUnits;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int64_t c = c0 + threadIdx.x + (int64_t)i * kThreads;
      if (c < a.n_out) {
        const int64_t s = a.src[c];
        if (s >= 0 && s < a.n_in) a.p_out[row * a.p_stride_out + c] = a.p_in[row * a.p_stride_in + s];
      }
    }
  }
}

}  // namespace
}  // namespace apack

using namespace apack;

extern "C" apack_status apack_compact_kv(int64_t n_out, const int32_t* src_rows, int64_t n_in, int32_t n_layers,
                                         const void* const* k_in, const void* const* v_in, void* const* k_out,
                                         void* const* v_out, int32_t hkv, int32_t d, apack_dtype dtype,
                                         int64_t head_stride_in, int64_t head_stride_out, const void* hidden_in,
                                         void* hidden_out, int32_t hidden_dim, const int32_t* pos_in,
                                         int32_t* pos_out, int32_t pos_rows, int64_t pos_stride_in,
                                         int64_t pos_stride_out, void* stream) {
  clear_error();
  APACK_CHECK(dtype_ok(dtype), APACK_E_DTYPE, "unknown dtype %d", (int)dtype);
  APACK_CHECK(n_out >= 0 && n_in >= 0, APACK_E_SHAPE, "negative row count");
  APACK_CHECK(n_out < (int64_t(1) << 31) && n_in < (int64_t(1) << 31), APACK_E_UNSUPPORTED,
              "row counts must be < 2^31");
  APACK_CHECK(n_layers >= 0 && n_layers <= kMaxTensors / 2, APACK_E_ARG, "n_layers must lie in [0, %d]",
              kMaxTensors / 2);
  APACK_CHECK(hidden_dim >= 0 && pos_rows >= 0, APACK_E_ARG, "negative hidden_dim or pos_rows");
  APACK_CHECK(n_out == 0 || src_rows, APACK_E_ARG, "src_rows is NULL");
  const size_t es = dtype_size(dtype);
  // v_in and v_out may both be NULL: then only the n_layers K planes move.
  const bool has_v = v_in != nullptr || v_out != nullptr;
  if (n_layers > 0) {
    APACK_CHECK(k_in && k_out, APACK_E_ARG, "K pointer tables must be non-NULL");
    APACK_CHECK(!has_v || (v_in && v_out), APACK_E_ARG, "v_in and v_out must both be NULL or both be set");
    APACK_CHECK(hkv > 0 && d > 0, APACK_E_SHAPE, "hkv and d must be positive");
    APACK_CHECK(head_stride_in >= n_in * d && head_stride_out >= n_out * d, APACK_E_SHAPE,
                "head strides must be >= rows * d");
  }
  const bool has_h = hidden_dim > 0;
  const bool has_p = pos_rows > 0;
  if (has_h) APACK_CHECK(hidden_in && hidden_out, APACK_E_ARG, "hidden_in/hidden_out must be non-NULL");
  if (has_p) {
    APACK_CHECK(pos_in && pos_out, APACK_E_ARG, "pos_in/pos_out must be non-NULL");
    APACK_CHECK(pos_stride_in >= n_in && pos_stride_out >= n_out, APACK_E_SHAPE,
                "position row strides must be >= rows");
  }
  // Alias checks: no output may overlap any input or another output.
  std::vector<std::pair<const void*, size_t>> ins, outs;
  const size_t kv_in_bytes = n_layers ? (size_t)((hkv - 1) * head_stride_in + n_in * d) * es : 0;
  const size_t kv_out_bytes = n_layers ? (size_t)((hkv - 1) * head_stride_out + n_out * d) * es : 0;
  for (int l = 0; l < n_layers; ++l) {
    APACK_CHECK(k_in[l] && k_out[l] && (!has_v || (v_in[l] && v_out[l])), APACK_E_ARG,
                "layer %d: NULL K/V pointer", l);
    ins.emplace_back(k_in[l], kv_in_bytes);
    outs.emplace_back(k_out[l], kv_out_bytes);
    if (has_v) {
      ins.emplace_back(v_in[l], kv_in_bytes);
      outs.emplace_back(v_out[l], kv_out_bytes);
    }
  }
  if (has_h) {
    ins.emplace_back(hidden_in, (size_t)n_in * hidden_dim * es);
    outs.emplace_back(hidden_out, (size_t)n_out * hidden_dim * es);
  }
  if (has_p) {
    ins.emplace_back(pos_in, (size_t)((pos_rows - 1) * pos_stride_in + n_in) * 4);
    outs.emplace_back(pos_out, (size_t)((pos_rows - 1) * pos_stride_out + n_out) * 4);
  }
  ins.emplace_back(src_rows, (size_t)n_out * 4);
  for (size_t i = 0; i < outs.size(); ++i) {
    for (auto& in : ins)
      APACK_CHECK(!overlaps(outs[i].first, outs[i].second, in.first, in.second), APACK_E_ALIAS,
                  "an output overlaps an input (compaction is out of place)");
    for (size_t j = i + 1; j < outs.size(); ++j)
      APACK_CHECK(!overlaps(outs[i].first, outs[i].second, outs[j].first, outs[j].second), APACK_E_ALIAS,
                  "two outputs overlap");
  }
  if (n_out == 0) return APACK_OK;

  // 16-byte units when every row, stride and base allows it, else 4 bytes.
  const int64_t kv_row_bytes = (int64_t)d * (int64_t)es;
  bool wide = true;
  auto al16 = [](const void* p) { return ((uintptr_t)p % 16) == 0; };
  if (n_layers) {
    wide &= kv_row_bytes % 16 == 0 && (head_stride_in * (int64_t)es) % 16 == 0 &&
            (head_stride_out * (int64_t)es) % 16 == 0;
    for (int l = 0; l < n_layers; ++l)
      wide &= al16(k_in[l]) && al16(k_out[l]) && (!has_v || (al16(v_in[l]) && al16(v_out[l])));
  }
  if (has_h) wide &= ((int64_t)hidden_dim * (int64_t)es) % 16 == 0 && al16(hidden_in) && al16(hidden_out);
  auto al4 = [](const void* p) { return ((uintptr_t)p % 4) == 0; };
  if (!wide) {
    APACK_CHECK(kv_row_bytes % 4 == 0 && ((int64_t)hidden_dim * (int64_t)es) % 4 == 0, APACK_E_UNSUPPORTED,
                "row sizes must be multiples of 4 bytes");
    for (int l = 0; l < n_layers; ++l)
      APACK_CHECK(al4(k_in[l]) && al4(k_out[l]) && (!has_v || (al4(v_in[l]) && al4(v_out[l]))), APACK_E_ARG,
                  "K/V pointers must be 4-byte aligned");
    if (has_h) APACK_CHECK(al4(hidden_in) && al4(hidden_out), APACK_E_ARG, "hidden must be 4-byte aligned");
  }
  const int64_t ub = wide ? 16 : 4;

  GatherArgs a;
  std::memset(&a, 0, sizeof a);
  a.src = src_rows;
  a.n_out = n_out;
  a.n_in = n_in;
  a.n_tensors = (has_v ? 2 : 1) * n_layers;
  a.heads = n_layers ? hkv : 1;
  if (n_layers) {
    a.row_units = kv_row_bytes / ub;
    a.hs_in = head_stride_in * (int64_t)es / ub;
    a.hs_out = head_stride_out * (int64_t)es / ub;
    a.kv_rows_per_item = std::max<int64_t>(1, kItemUnits / a.row_units);
    a.row_magic = div_magic(a.row_units);
    a.kv_items_per_plane = (n_out + a.kv_rows_per_item - 1) / a.kv_rows_per_item;
    a.kv_items = a.kv_items_per_plane * a.n_tensors * hkv;
    for (int l = 0; l < n_layers; ++l) {
      if (has_v) {
        a.in[2 * l] = k_in[l];
        a.in[2 * l + 1] = v_in[l];
        a.out[2 * l] = k_out[l];
        a.out[2 * l + 1] = v_out[l];
      } else {
        a.in[l] = k_in[l];
        a.out[l] = k_out[l];
      }
    }
    APACK_CHECK(a.row_units <= kItemUnits, APACK_E_UNSUPPORTED, "K/V rows longer than %d bytes",
                (int)(kItemUnits * ub));
  }
  if (has_h) {
    a.h_in = hidden_in;
    a.h_out = hidden_out;
    a.h_row_units = (int64_t)hidden_dim * (int64_t)es / ub;
    APACK_CHECK(a.h_row_units <= kItemUnits, APACK_E_UNSUPPORTED, "hidden rows longer than %d bytes",
                (int)(kItemUnits * ub));
    a.h_rows_per_item = std::max<int64_t>(1, kItemUnits / a.h_row_units);
    a.h_row_magic = div_magic(a.h_row_units);
    a.h_items = (n_out + a.h_rows_per_item - 1) / a.h_rows_per_item;
  }
  if (has_p) {
    a.p_in = pos_in;
    a.p_out = pos_out;
    a.p_rows = pos_rows;
    a.p_stride_in = pos_stride_in;
    a.p_stride_out = pos_stride_out;
    a.p_items_per_row = (n_out + kItemUnits - 1) / kItemUnits;
    a.p_items = a.p_items_per_row * pos_rows;
  }
  const int64_t items = a.kv_items + a.h_items + a.p_items;
  if (items == 0) return APACK_OK;
  APACK_CHECK(items < (int64_t(1) << 31), APACK_E_UNSUPPORTED, "too many work items");
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (wide)
    hipLaunchKernelGGL(k_gather<u32x4>, dim3((unsigned)items), dim3(kThreads), 0, hs, a);
  else
    hipLaunchKernelGGL(k_gather<uint32_t>, dim3((unsigned)items), dim3(kThreads), 0, hs, a);
  return launch_status("k_gather");
}
