// Integrated score and flat top-B (Eq. modal_scoring and Sec. integrated
// scoring of the paper), one work-group per (unit, sequence):
//   S = A on text tokens, S = M * (A + alpha * Phi) on visual tokens,
//   I_keep = the B tokens first in (S descending, index ascending) order,
//   written in ascending token order.
// S is turned into a descending order key once, the B-th key is found by a
// four-pass radix select, and one ordered pass with two work-group scans
// resolves ties at the threshold by lowest index and compacts the survivors.
#include "block_select.h"
#include "stlite_internal.h"

namespace stlite {
namespace {

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectArgs a) {
  __shared__ SelectShared sh;
  const Layout& lay = a.lay;
  const int s = blockIdx.x, unit = blockIdx.y, tid = threadIdx.x;
  const int32_t seq_start = lay.cu_seqlens[s], seq_end = lay.cu_seqlens[s + 1];
  const int32_t L = seq_end - seq_start;
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  const int32_t kept_base = lay.cu_budget[s];
  const int32_t B = lay.cu_budget[s + 1] - kept_base;
  const size_t ubase = size_t(unit) * lay.total_tokens;
  const float* A = a.a_base + ubase;
  const float* phi = a.phi ? a.phi + ubase : nullptr;
  const uint8_t* gate = a.gate ? a.gate + ubase : nullptr;
  float* score = a.score ? a.score + ubase : nullptr;
  uint32_t* keys = a.keys + ubase + seq_start;  // keys[j] for token seq_start + j
  int32_t* kept = a.kept + size_t(unit) * lay.total_budget + kept_base;
  const float alpha = a.alpha;

  // Scores, segment by segment (text gap, frame, ..., trailing text).
  int32_t prev = seq_start;
  for (int32_t f = f0; f <= f1; ++f) {
    const bool is_frame = f < f1;
    const int32_t off = is_frame ? lay.frame_meta[3 * f] : seq_end;
    for (int32_t j = prev + tid; j < off; j += kSelThreads) {
      const float S = A[j];
      if (score) score[j] = S;
      keys[j - seq_start] = ~order_key(S);
    }
    if (is_frame) {
      const int32_t n = lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
      for (int32_t j = off + tid; j < off + n; j += kSelThreads) {
        const float x = phi ? fmaf(alpha, phi[j], A[j]) : A[j];
        const float S = (gate && gate[j] == 0) ? 0.0f : x;
        if (score) score[j] = S;
        keys[j - seq_start] = ~order_key(S);
      }
      prev = off + n;
    }
  }
  if (B == 0) return;
  __syncthreads();

  int32_t need = 0;
  uint32_t T = 0xffffffffu;
  if (B < L) T = block_radix_select(keys, L, B, sh, &need);
  else need = L;  // keep everything: every key is <= T

  int32_t running_eq = 0, running_kept = 0;
  for (int32_t base = 0; base < L; base += kSelThreads) {
    const int32_t j = base + tid;
    const bool in = j < L;
    const uint32_t key = in ? keys[j] : 0xffffffffu;
    const bool eq = in && key == T;
    int32_t eq_tot, kept_tot;
    const int32_t eq_incl = block_inclusive_scan(eq ? 1 : 0, sh.wave_tot, &eq_tot);
    const bool take = (in && key < T) || (eq && running_eq + eq_incl - 1 < need);
    const int32_t k_incl = block_inclusive_scan(take ? 1 : 0, sh.wave_tot2, &kept_tot);
    if (take && running_kept + k_incl - 1 < B) kept[running_kept + k_incl - 1] = seq_start + j;
    running_eq += eq_tot;
    running_kept += kept_tot;
  }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(select_kernel, dim3(a.lay.n_seqs, a.lay.n_units), dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
