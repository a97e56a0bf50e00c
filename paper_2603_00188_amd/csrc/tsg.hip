// Trajectory-aware Semantic Gating (Sec. TSG of the paper).
//
//   rho_i = max_{j in current frame} cos(k_i, k_j)   for historical visual i
//   m = min(B, |pool|); the gate admits the m historical tokens first in
//   (rho ascending, index ascending) order (Eqs. budget_threshold and
//   temporal_mask in rank form); current frame and text get gate 1.  The
//   selection itself is in gate.hip.
//
// rho is a dense N_hist x N_cur x 128 contraction: bf16 MFMA tiles with the
// historical rows resident in VGPRs (A operand, 256 rows per work-group) and
// the current frame streamed through LDS in 64-key tiles (B operand).  The
// epilogue never stores the logits: each lane scales its column by the key's
// inverse norm and keeps a running row max; 16-lane butterflies finish the max.
//
// The similarity-metric ablation swaps the cosine for the dot product (the
// running max of the raw products) or the negative L2 distance: since
// -||a - b||^2 = 2 a.b - ||b||^2 - ||a||^2, the running max of 2 a.b - ||b||^2
// (one fma per product, as the cosine's one multiply) gives the smallest
// distance, and rho = -sqrt(max(||a||^2 - max, 0)), snapped to 0 when the
// squared distance is at most 1e-5 ||a||^2.
//
// The fixed-threshold control of the component-necessity study replaces the
// rank gate with gate = 1[rho <= tau] for a fixed tau.
#include <algorithm>

#include "stlite_internal.h"
#include "tile_lds.h"

namespace stlite {
namespace {


constexpr float kSnap = 1.0f - 1.0e-4f;
constexpr float kL2Snap = 1.0e-5f;

__device__ inline int32_t frame_size(const Layout& lay, int32_t f) {
  return lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
}

__device__ inline int32_t hist_count(const Layout& lay, int32_t s) {
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  int32_t n = 0;
  for (int32_t f = f0; f + 1 < f1; ++f) n += frame_size(lay, f);
  return n;
}

// Plan of the TSG pass.  Work-groups 0 .. n_seqs-1: per sequence, the 256-row
// block descriptors of the rho GEMM.  Work-groups n_seqs + f: the historical
// token table entries of frame f (frames in order, row-major inside a frame),
// unless f is its sequence's current frame.
__global__ __launch_bounds__(256) void tsg_plan_kernel(GateArgs a) {
  const Layout& lay = a.lay;
  if (int32_t(blockIdx.x) < lay.n_seqs) {
    const int s = blockIdx.x;
    int32_t hist_base = 0, blk_base = 0;
    for (int32_t t = 0; t < s; ++t) {
      const int32_t n = hist_count(lay, t);
      hist_base += n;
      blk_base += (n + kRhoRows - 1) / kRhoRows;
    }
    const int32_t n_hist = hist_count(lay, s);
    const int32_t nb = (n_hist + kRhoRows - 1) / kRhoRows;
    for (int32_t b = threadIdx.x; b < nb; b += blockDim.x) a.blocks[blk_base + b] = HistBlock{s, b, n_hist, hist_base};
    return;
  }
  const int32_t f = int32_t(blockIdx.x) - lay.n_seqs;
  int32_t s = 0;  // sequence of frame f
  while (lay.cu_frames[s + 1] <= f) ++s;
  if (f == lay.cu_frames[s + 1] - 1) return;  // current frame: not historical
  int32_t h = 0;  // historical rows before frame f, over all sequences
  for (int32_t t = 0; t < s; ++t) h += hist_count(lay, t);
  for (int32_t g = lay.cu_frames[s]; g < f; ++g) h += frame_size(lay, g);
  const int32_t off = lay.frame_meta[3 * f], n = frame_size(lay, f);
  for (int32_t j = threadIdx.x; j < n; j += blockDim.x) a.hist_tok[h + j] = off + j;
}

// gate = 1 on every token (the selection then decides the historical ones)
// and rho = 0 everywhere; either pointer may be null.  (The rho call zeroes
// only the tokens that are not historical, with rho_zero_kernel.)
__global__ __launch_bounds__(256) void gate_fill_kernel(GateArgs a, size_t n) {
  const size_t stride = size_t(gridDim.x) * blockDim.x;
  const size_t i0 = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  uint8_t* gate = a.gate;
  float* rho = a.rho_zero_fill;
  const bool vec = (reinterpret_cast<uintptr_t>(gate) & 3) == 0 && (reinterpret_cast<uintptr_t>(rho) & 15) == 0;
  size_t done = 0;
  if (vec) {
    const size_t n4 = n / 4;
    for (size_t i = i0; i < n4; i += stride) {
      if (gate) reinterpret_cast<uint32_t*>(gate)[i] = 0x01010101u;
      if (rho) reinterpret_cast<float4*>(rho)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    done = 4 * n4;
  }
  for (size_t i = done + i0; i < n; i += stride) {
    if (gate) gate[i] = 1;
    if (rho) rho[i] = 0.0f;
  }
}

// rho = 0 on the tokens that are not historical (text and each sequence's
// current frame); the rho pass writes every historical token.  Work-group
// (g, unit) covers token run g (token_run, current frames included).
__global__ __launch_bounds__(256) void rho_zero_kernel(GateArgs a) {
  const Layout& lay = a.lay;
  float* rho = a.rho_zero_fill + size_t(blockIdx.y) * lay.total_tokens;
  int32_t b, e;
  token_run(lay, int32_t(blockIdx.x), true, &b, &e);
  for (int32_t j = b + int32_t(threadIdx.x); j < e; j += blockDim.x) rho[j] = 0.0f;
}

__device__ inline float sumsq8(uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float lo = __uint_as_float(w[j] << 16), hi = __uint_as_float(w[j] & 0xffff0000u);
    s = fmaf(lo, lo, s);
    s = fmaf(hi, hi, s);
  }
  return s;
}

// Column factors of the current-frame keys: rn[unit][token] = 1/||k|| (0 for a
// zero key), or -||k||^2 under the negative L2 distance.  Work-group
// (x, seq, unit) covers keys 64 x .. 64 x + 63 of the sequence's current
// frame, 16 lanes per key.
template <int SIM>
__global__ __launch_bounds__(256) void cur_norms_kernel(RhoArgs a) {
  const int s = blockIdx.y, unit = blockIdx.z;
  const Layout& lay = a.lay;
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  if (f1 - f0 < 2) return;  // no history: nothing reads the current-frame norms
  const int32_t off = lay.frame_meta[3 * (f1 - 1)];
  const int32_t n = min(frame_size(lay, f1 - 1), int32_t(blockIdx.x + 1) * 64);
  const uint16_t* kunit = a.k + size_t(unit) * lay.total_tokens * kHeadDim;
  float* rn = a.rn_cur + size_t(unit) * lay.total_tokens;
  // 16 groups of 16 lanes, four keys per group: all four loads first.
  const int group = threadIdx.x >> 4, gl = threadIdx.x & 15;
  const int32_t j0 = int32_t(blockIdx.x) * 64 + group;
  uint4 v[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int32_t j = j0 + 16 * q;
    v[q] = j < n ? *reinterpret_cast<const uint4*>(kunit + size_t(off + j) * kHeadDim + gl * 8) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int32_t j = j0 + 16 * q;
    float ss = sumsq8(v[q]);
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o);
    if (gl == 0 && j < n) rn[off + j] = SIM == kSimNegL2 ? -ss : (ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f);
  }
}

// One work-group = 4 waves x 64 historical rows (the MFMA A operand, resident
// in VGPRs).  The current frame streams through a three-stage ring of LDS
// tiles filled by direct memory->LDS DMA: tile n+2 is in flight while tile n
// feeds the matrix cores.  Key slots past the end of the frame repeat the
// frame's last key, which leaves every row max unchanged and needs no mask.
// The three stages are distinct LDS arrays and the loop is unrolled by three,
// so that every tile read has a compile-time LDS address.
template <int SIM>
__global__ __launch_bounds__(256, 2) void rho_kernel(RhoArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks0[kTileElems], ks1[kTileElems], ks2[kTileElems];
  __shared__ __attribute__((aligned(16))) float rn0[kTileKeys], rn1[kTileKeys], rn2[kTileKeys];
  __shared__ int32_t tok_s[kRhoRows];
  __shared__ float rnrow_s[kRhoRows];
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const HistBlock hb = a.blocks[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t last = lay.cu_frames[hb.seq + 1] - 1;
  const int32_t cur_off = lay.frame_meta[3 * last];
  const int32_t n_cur = frame_size(lay, last);
  const int32_t ntiles = (n_cur + kTileKeys - 1) / kTileKeys;
  const uint16_t* kunit = a.k + size_t(unit) * lay.total_tokens * kHeadDim;
  const uint16_t* kcur = kunit + size_t(cur_off) * kHeadDim;
  const float* rn_cur = a.rn_cur + size_t(unit) * lay.total_tokens + cur_off;

  const TileDma<4> dma;
  const __amdgpu_buffer_rsrc_t rn_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(rn_cur), 0, n_cur * 4, kBufferFlags);
  // Tile n: 4 key wave-loads per wave, plus the 64 inverse norms on wave 0 (a
  // frame's norms are one small buffer; slots past its end repeat the last).
  auto issue = [&](int32_t n, uint16_t* tile, float* rn) {
    dma.issue(kcur, n * kTileKeys, n_cur - 1, tile);
    if (wave == 0) {
      uint32_t dst = uint32_t(reinterpret_cast<uintptr_t>(rn));
      asm volatile("" : "+s"(dst));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rn_rsrc, (lds_void_t)(uintptr_t)dst, 4,
                                               uint32_t(min(n * kTileKeys + lane, n_cur - 1)) * 4u, 0, 0, 0);
    }
  };
  issue(0, ks0, rn0);
  if (ntiles > 1) issue(1, ks1, rn1);

  // Historical rows: A operand (row = lane & 15 of each 16-row block).
  int32_t tok[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int32_t h = hb.hb * kRhoRows + wave * 64 + b * 16 + (lane & 15);
    tok[b] = h < hb.n_hist ? a.hist_tok[hb.hist_base + h] : -1;
  }
  bf16x8_t ha[4][4];
  float ss[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    uint4 v[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      v[kk] = tok[b] >= 0 ? *reinterpret_cast<const uint4*>(kunit + size_t(tok[b]) * kHeadDim + kk * 32 + (lane >> 4) * 8)
                          : make_uint4(0, 0, 0, 0);
    ss[b] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      ss[b] += sumsq8(v[kk]);
      ha[b][kk] = __builtin_bit_cast(bf16x8_t, v[kk]);
    }
  }
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    float x = ss[b] + __shfl_xor(ss[b], 16);
    x += __shfl_xor(x, 32);
    if (lane < 16) {
      tok_s[wave * 64 + b * 16 + lane] = tok[b];
      // cosine: 1/||a||; -L2: ||a||^2; unused by the dot product
      rnrow_s[wave * 64 + b * 16 + lane] = SIM == kSimNegL2 ? x : (x > 0.0f ? 1.0f / sqrtf(x) : 0.0f);
    }
  }

  float runmax[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) runmax[b][i] = -INFINITY;

  // Ping-pong inside the wave.  A tile is two halves (16-key sub-tiles 0-1 and
  // 2-3); the 32 MFMAs of one half are issued among the scale-and-max
  // instructions of the other half (carried across the tile boundary), and
  // the B operand is read from LDS one k-step ahead of its MFMAs.
  // The B fragments of the tile's eight k-steps (g = 4 h + kk: half h, k-step
  // kk) go through a three-slot register ring, read two k-steps ahead of
  // their MFMAs -- including the first two k-steps of the second half, which
  // are read under the first half's MFMAs.
  bf16x8_t kb[3][2];
  auto read_b = [&](const uint16_t* tile, int g) {
#pragma unroll
    for (int t = 0; t < 2; ++t) kb[g % 3][t] = tile_b_operand(tile, 2 * (g / 4) + t, g % 4);
  };
  auto mfma_half = [&](const uint16_t* tile, int h, f32x4_t (&acc)[4][2]) {
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int t = 0; t < 2; ++t) acc[b][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int g = 4 * h + kk;
      if (g + 2 < 8) read_b(tile, g + 2);
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int t = 0; t < 2; ++t)
          acc[b][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[b][kk], kb[g % 3][t], acc[b][t], 0, 0, 0);
    }
  };
  auto column = [&](float x, float rn) {
    if constexpr (SIM == kSimCosine) return x * rn;
    else if constexpr (SIM == kSimDot) return x;
    else return fmaf(x, 2.0f, rn);
  };
  auto max_half = [&](const f32x4_t (&acc)[4][2], float rn0, float rn1) {
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        runmax[b][i] =
            __builtin_fmaxf(__builtin_fmaxf(runmax[b][i], column(acc[b][0][i], rn0)), column(acc[b][1][i], rn1));
  };
  // Per half: B fragments read under the MFMAs of earlier k-steps, 3 VALU
  // (scale and max of the other half) per 2 MFMAs.
  auto interleave = [&](int h) {
    if (h == 0) __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // k-steps 0 and 1
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (4 * h + kk + 2 < 8) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // read ahead
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // 2 MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // 3 VALU
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  f32x4_t accA[4][2], accB[4][2];
  // Before the first tile the "previous second half" contributes -inf to every max.
  float rnB0 = 1.0f, rnB1 = 1.0f;  // norms of the previous tile's second half
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int t = 0; t < 2; ++t) accB[b][t] = f32x4_t{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  // One tile: wait for its DMA (at most tile n+1's loads stay outstanding),
  // launch the DMA of tile n+2 into the stage read in the previous step.
  auto step = [&](int32_t n, const uint16_t* tile, const float* rn, uint16_t* nxt, float* nxt_rn) {
    if (n + 1 < ntiles) {
      if (wave == 0) wait_vmcnt<5>(); else wait_vmcnt<4>();
    } else {
      wait_vmcnt<0>();
    }
    barrier_lds();
    const float rnA0 = rn[0 * 16 + (lane & 15)], rnA1 = rn[1 * 16 + (lane & 15)];
    const float rnN0 = rn[2 * 16 + (lane & 15)], rnN1 = rn[3 * 16 + (lane & 15)];
    read_b(tile, 0);
    read_b(tile, 1);
    mfma_half(tile, 0, accA);
    max_half(accB, rnB0, rnB1);
    interleave(0);
    if (n + 2 < ntiles) issue(n + 2, nxt, nxt_rn);
    mfma_half(tile, 1, accB);
    max_half(accA, rnA0, rnA1);
    interleave(1);
    rnB0 = rnN0;
    rnB1 = rnN1;
  };
  for (int32_t n = 0; n < ntiles; n += 3) {
    step(n, ks0, rn0, ks2, rn2);
    if (n + 1 < ntiles) step(n + 1, ks1, rn1, ks0, rn0);
    if (n + 2 < ntiles) step(n + 2, ks2, rn2, ks1, rn1);
  }
  max_half(accB, rnB0, rnB1);

  float* rho = a.rho + size_t(unit) * lay.total_tokens;
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = runmax[b][i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      if ((lane & 15) == 0) {
        const int r = wave * 64 + b * 16 + (lane >> 4) * 4 + i;
        const int32_t t = tok_s[r];
        if (t >= 0) {
          float x;
          if constexpr (SIM == kSimCosine) {
            x = fminf(fmaxf(mx * rnrow_s[r], -1.0f), 1.0f);
            if (x >= kSnap) x = 1.0f;
          } else if constexpr (SIM == kSimDot) {
            x = mx;
          } else {
            const float n = rnrow_s[r];
            float d2 = fmaxf(n - mx, 0.0f);
            if (d2 <= kL2Snap * n) d2 = 0.0f;
            x = -sqrtf(d2);
          }
          rho[t] = x + 0.0f;
        }
      }
    }
}

// Fixed-threshold gate of frame blockIdx.x in unit blockIdx.y: every token of a
// historical frame gets 1[rho <= tau]; the current frame keeps the 1 of the fill.
__global__ __launch_bounds__(256) void fixed_gate_kernel(GateArgs a, float tau) {
  const Layout& lay = a.lay;
  const int32_t f = blockIdx.x;
  int32_t lo = 0, hi = lay.n_seqs - 1;
  while (lo < hi) {  // the sequence whose frames f lies in
    const int32_t mid = (lo + hi + 1) >> 1;
    if (lay.cu_frames[mid] <= f) lo = mid; else hi = mid - 1;
  }
  if (f == lay.cu_frames[lo + 1] - 1) return;  // current frame
  const size_t base = size_t(blockIdx.y) * lay.total_tokens;
  const int32_t off = lay.frame_meta[3 * f], n = frame_size(lay, f);
  for (int32_t j = threadIdx.x; j < n; j += blockDim.x) a.gate[base + off + j] = a.rho[base + off + j] <= tau ? 1 : 0;
}

}  // namespace

hipError_t launch_gate_prologue(const GateArgs& g, hipStream_t stream) {
  hipLaunchKernelGGL(tsg_plan_kernel, dim3(g.lay.n_seqs + g.lay.n_frames), dim3(256), 0, stream, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (g.gate) {
    GateArgs fill = g;
    fill.rho_zero_fill = nullptr;
    const size_t n = size_t(g.lay.n_units) * g.lay.total_tokens;
    const unsigned blocks = unsigned(std::min<size_t>((n / 4 + 255) / 256 + 1, 8192));
    hipLaunchKernelGGL(gate_fill_kernel, dim3(blocks), dim3(256), 0, stream, fill, n);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (g.rho_zero_fill && g.lay.n_units > 0)
    hipLaunchKernelGGL(rho_zero_kernel, dim3(g.lay.n_frames + g.lay.n_seqs, g.lay.n_units), dim3(256), 0, stream, g);
  return hipGetLastError();
}

hipError_t launch_tsg_threshold(const GateArgs& g, hipStream_t stream) { return launch_gate_select(g, stream); }

hipError_t launch_tsg_rho(const RhoArgs& r, const GateArgs& g, hipStream_t stream) {
  hipError_t e = launch_gate_prologue(g, stream);
  if (e != hipSuccess) return e;
  const dim3 norm_grid((std::max(r.max_cur, 1) + 63) / 64, r.lay.n_seqs, r.lay.n_units);
  const dim3 rho_grid(r.total_hist_blocks, r.lay.n_units);
  switch (r.sim) {
    case kSimCosine:
      hipLaunchKernelGGL(cur_norms_kernel<kSimCosine>, norm_grid, dim3(256), 0, stream, r);
      if (r.total_hist_blocks > 0) hipLaunchKernelGGL(rho_kernel<kSimCosine>, rho_grid, dim3(256), 0, stream, r);
      break;
    case kSimDot:  // the dot product needs no column factors
      if (r.total_hist_blocks > 0) hipLaunchKernelGGL(rho_kernel<kSimDot>, rho_grid, dim3(256), 0, stream, r);
      break;
    case kSimNegL2:
      hipLaunchKernelGGL(cur_norms_kernel<kSimNegL2>, norm_grid, dim3(256), 0, stream, r);
      if (r.total_hist_blocks > 0) hipLaunchKernelGGL(rho_kernel<kSimNegL2>, rho_grid, dim3(256), 0, stream, r);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_tsg_fixed_gate(const GateArgs& g, float tau, hipStream_t stream) {
  const size_t n = size_t(g.lay.n_units) * g.lay.total_tokens;
  const unsigned blocks = unsigned(std::min<size_t>((n / 4 + 255) / 256 + 1, 8192));
  hipLaunchKernelGGL(gate_fill_kernel, dim3(blocks), dim3(256), 0, stream, g, n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.lay.n_frames == 0 || g.lay.n_units == 0) return e;
  hipLaunchKernelGGL(fixed_gate_kernel, dim3(g.lay.n_frames, g.lay.n_units), dim3(256), 0, stream, g, tau);
  return hipGetLastError();
}

hipError_t launch_tsg_gate(const RhoArgs& r, const GateArgs& g, hipStream_t stream) {
  GateArgs pro = g;
  pro.gate = nullptr;  // the gate kernel writes every gate byte itself
  hipError_t e = launch_tsg_rho(r, pro, stream);
  if (e != hipSuccess) return e;
  return launch_gate_select(g, stream);
}

}  // namespace stlite
