// Cache compaction (the compression procedure's result K' = K[I_keep],
// V' = V[I_keep]): a coalesced gather of 256-byte bf16 rows.  Sixteen lanes
// move one row with 16-byte loads and stores; a work-group moves 64 rows of K
// and of V.  The stream touches each byte once, so loads and stores bypass
// the caches' retention (non-temporal).
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kRowsPerGroup = 64;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void compact_kernel(CompactArgs a) {
  constexpr int kPer = kRowsPerGroup / 16;  // rows per 16-lane group
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const int64_t j0 = int64_t(blockIdx.x) * kRowsPerGroup;
  const int sub = threadIdx.x >> 4, part = threadIdx.x & 15;
  const size_t ubase = size_t(unit) * lay.total_tokens;
  const size_t obase = size_t(unit) * lay.total_budget;
  const size_t kbase = size_t(a.kept_per_layer ? unit / lay.n_kv_heads : unit) * lay.total_budget;
  // All of a thread's loads are issued before its stores, so that each lane
  // keeps 2 * kPer 16-byte reads in flight.
  int32_t tok[kPer];
  bool row_ok[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int64_t j = j0 + r * 16 + sub;
    row_ok[r] = j < lay.total_budget;
    tok[r] = row_ok[r] ? a.kept[kbase + j] : -1;
  }
  // Loads are unconditional (an out-of-range index reads row 0 and is stored
  // as zeros), so that no branch forces a wait between them.
  u32x4_t kv[kPer], vv[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const bool ok = tok[r] >= 0 && tok[r] < lay.total_tokens;
    const size_t src = (ubase + size_t(ok ? tok[r] : 0)) * kHeadDim + part * 8;
    kv[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.k + src));
    vv[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.v + src));
  }
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const bool ok = tok[r] >= 0 && tok[r] < lay.total_tokens;
    if (!ok) {
      kv[r] = u32x4_t{0u, 0u, 0u, 0u};
      vv[r] = u32x4_t{0u, 0u, 0u, 0u};
    }
    if (!row_ok[r]) continue;
    const size_t dst = (obase + size_t(j0 + r * 16 + sub)) * kHeadDim + part * 8;
    __builtin_nontemporal_store(kv[r], reinterpret_cast<u32x4_t*>(a.k_out + dst));
    __builtin_nontemporal_store(vv[r], reinterpret_cast<u32x4_t*>(a.v_out + dst));
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.lay.total_budget + kRowsPerGroup - 1) / kRowsPerGroup;
  hipLaunchKernelGGL(compact_kernel, dim3(uint32_t(blocks), a.lay.n_units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
