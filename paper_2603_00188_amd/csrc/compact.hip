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
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const int64_t j0 = int64_t(blockIdx.x) * kRowsPerGroup;
  const int sub = threadIdx.x >> 4, part = threadIdx.x & 15;
  const size_t ubase = size_t(unit) * lay.total_tokens;
  const size_t obase = size_t(unit) * lay.total_budget;
#pragma unroll
  for (int r = 0; r < kRowsPerGroup; r += 16) {
    const int64_t j = j0 + r + sub;
    if (j >= lay.total_budget) break;
    const int32_t tok = a.kept[obase + j];
    u32x4_t kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
    if (tok >= 0 && tok < lay.total_tokens) {
      const size_t src = (ubase + size_t(tok)) * kHeadDim + part * 8;
      kv = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.k + src));
      vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.v + src));
    }
    const size_t dst = (obase + size_t(j)) * kHeadDim + part * 8;
    __builtin_nontemporal_store(kv, reinterpret_cast<u32x4_t*>(a.k_out + dst));
    __builtin_nontemporal_store(vv, reinterpret_cast<u32x4_t*>(a.v_out + dst));
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.lay.total_budget + kRowsPerGroup - 1) / kRowsPerGroup;
  hipLaunchKernelGGL(compact_kernel, dim3(uint32_t(blocks), a.lay.n_units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
