// Rank form of the TSG gate (Eqs. budget_threshold and temporal_mask of the
// paper): per (sequence, unit), m = min(B, N_hist) historical tokens are
// admitted, those first in (rho ascending, index ascending) order; tau_red is
// the rho of the last one admitted.  The selection is the exact k-selection of
// segsel.h over the keys order_key(rho).
#include "segsel.h"
#include "segsel_resident.h"
#include "segsel_split.h"
#include "stlite_internal.h"

namespace stlite {
namespace {

__device__ inline int32_t frame_size(const Layout& lay, int32_t f) {
  return lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
}

// Rank gate of one (sequence, unit) segment: the keys are order_key(rho) on
// historical tokens (a NaN rho is kept below the never-selected key) and
// kSelNever elsewhere; k = m = min(B, N_hist).  Every gate byte of the
// sequence is written: 1 on text and the current frame, 1 on the m admitted
// historical tokens and 0 on the others.
template <bool LDS>
struct GateProd {
  __amdgpu_buffer_rsrc_t rho;   // the segment's rho (out-of-range lanes read 0)
  __amdgpu_buffer_rsrc_t gate;  // the segment's gate bytes
  SeqFrames<LDS> fr;

  __device__ int32_t cursor(const SelCtx& c, int32_t i) const { return __builtin_amdgcn_readfirstlane(fr.find(c.s0 + i)); }

  struct Raw {
    uint32_t hist;  // bit j: token j of the step is historical
    float r[kSelJ];
  };

  __device__ void fetch(const SelCtx& c, int32_t base, int32_t lane, int32_t& cur, Raw& w) const {
    const StepFrames st = step_frames(fr, cur, c.s0 + base, 64 * kSelJ);
    const int u = st.n >= 0 ? st.uniform(c.s0 + base, 64 * kSelJ) : -1;
    w.hist = 0u;
    if (u >= 0) {
      w.hist = u == kHist ? (1u << kSelJ) - 1u : 0u;
    } else if (st.n >= 0) {
#pragma unroll
      for (int j = 0; j < kSelJ; ++j) w.hist |= (st.cls(c.s0 + base + 64 * j + lane) == kHist ? 1u : 0u) << j;
    } else {
#pragma unroll
      for (int j = 0; j < kSelJ; ++j) w.hist |= (tok_class_search(fr, c.s0 + base + 64 * j + lane) == kHist ? 1u : 0u) << j;
    }
#pragma unroll
    for (int j = 0; j < kSelJ; ++j)
      w.r[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rho, (base + 64 * j + lane) * 4, 0, 0));
  }

  __device__ void finish(const SelCtx&, int32_t base, int32_t lane, int32_t hi, const Raw& w,
                         uint32_t (&key)[kSelJ]) const {
#pragma unroll
    for (int j = 0; j < kSelJ; ++j) {
      const bool h = ((w.hist >> j) & 1u) && base + 64 * j + lane < hi;
      key[j] = h ? min(order_key(w.r[j]), kSelKeyMax) : kSelNever;
    }
  }

  __device__ void emit(const SelCtx&, int32_t i, uint32_t key, bool take, int32_t) const {
    __builtin_amdgcn_raw_buffer_store_b8(uint8_t((key == kSelNever || take) ? 1 : 0), gate, i, 0, 0);
  }
};

__device__ inline void gate_buffers(const GateArgs& a, const SelCtx& c, __amdgpu_buffer_rsrc_t& rho,
                                    __amdgpu_buffer_rsrc_t& gate) {
  const size_t seg0 = c.ubase + size_t(c.s0);
  rho = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.rho) + seg0, 0, c.n * 4, kBufferFlags);
  gate = __builtin_amdgcn_make_buffer_rsrc(a.gate + seg0, 0, c.n, kBufferFlags);
}

// Work-group (part, seq, unit): keys of one part of a segment; k = min(B, N_hist).
// LDS: every sequence has at most kSelFrames frames (their ranges go to LDS).
template <bool LDS>
__global__ __launch_bounds__(kSelThreads) void gate_produce_kernel(GateArgs a) {
  __shared__ SelShared sh;
  const Layout& lay = a.lay;
  SelCtx c = sel_ctx(lay);
  GateProd<LDS> p{};
  gate_buffers(a, c, p.rho, p.gate);
  p.fr = load_frames<LDS>(sh, lay, c.seq);
  int32_t nh = 0;  // N_hist: every frame of the sequence but the last
  for (int32_t f = threadIdx.x; f + 1 < p.fr.nf; f += kSelThreads) nh += frame_size(lay, p.fr.f0 + f);
  nh = wave_sum(nh);
  if ((threadIdx.x & 63) == 0) sh.red[threadIdx.x >> 6] = nh;
  __syncthreads();
  int32_t n_hist = 0;
  for (int w = 0; w < kSelWaves; ++w) n_hist += sh.red[w];
  c.k = min(lay.cu_budget[c.seq + 1] - lay.cu_budget[c.seq], n_hist);
  sel_produce(p, sh, a.sel, lay, c);
}

// Work-group (part, seq, unit): gate bytes of one part of a segment; part 0
// writes tau.
__global__ __launch_bounds__(kSelThreads) void gate_emit_kernel(GateArgs a) {
  __shared__ SelShared sh;
  const Layout& lay = a.lay;
  SelCtx c = sel_ctx(lay);
  GateProd<false> p{};  // the emit pass reads keys only
  gate_buffers(a, c, p.rho, p.gate);
  const uint32_t T = sel_emit(p, sh, a.sel, lay, c);
  if (a.tau && c.part == 0 && threadIdx.x == 0)
    a.tau[size_t(blockIdx.z) * lay.n_seqs + c.seq] = c.k > 0 ? order_key_value(T) : __builtin_nanf("");
}

// The rank gate of one segment held by one work-group (segsel_resident.h).
struct GateRes {
  static constexpr int kGroup = 1;      // tiles a classifying wave loads at once (segsel_split.h)
  static constexpr bool kDirect = true;  // the splitter path writes the gate bytes directly
  __amdgpu_buffer_rsrc_t rho;
  __amdgpu_buffer_rsrc_t gate;
  bool needs_class;
  bool aligned;  // the segment's gate bytes start 4-byte aligned

  struct Raw {
    float r[4];
  };

  __device__ void load(int32_t base, Raw& w) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w.r[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rho, (base + 64 * e + lane) * 4, 0, 0));
  }

  __device__ void keys(int32_t base, const int (&cls)[4], int32_t hi, const Raw& w, uint32_t (&key)[4]) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      key[e] = (cls[e] == kHist && base + 64 * e + lane < hi) ? min(order_key(w.r[e]), kSelKeyMax) : kSelNever;
  }

  __device__ void emit(int32_t i, int cls, bool take, int32_t) const {
    __builtin_amdgcn_raw_buffer_store_b8(uint8_t((cls != kHist || take) ? 1 : 0), gate, i, 0, 0);
  }

  // Whether a token of class cls can be selected (segsel_split.h).
  __device__ bool selectable(int cls) const { return cls == kHist; }

  // keys() for a whole tile of one class (cls, wave-uniform) inside the segment.
  __device__ void keys_uniform(int32_t, int cls, const Raw& w, uint32_t (&key)[4]) const {
#pragma unroll
    for (int e = 0; e < 4; ++e) key[e] = cls == kHist ? min(order_key(w.r[e]), kSelKeyMax) : kSelNever;
  }

  // The splitter path (segsel_split.h): one token's input and key, and the
  // gate byte from its code (never selected = not historical).
  struct Raw1 {
    float r;
  };

  __device__ void load1(int32_t i, Raw1& w) const {
    w.r = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rho, i * 4, 0, 0));
  }
  __device__ void load1_rest(int32_t, int, Raw1&) const {}

  __device__ uint32_t key1(const Raw1& w, int cls) const {
    return cls == kHist ? min(order_key(w.r), kSelKeyMax) : kSelNever;
  }

  __device__ void emit_code(int32_t i, bool never, bool take, int32_t) const {
    __builtin_amdgcn_raw_buffer_store_b8(uint8_t((never || take) ? 1 : 0), gate, i, 0, 0);
  }

  __device__ void put_byte(int32_t i, uint8_t b) const { __builtin_amdgcn_raw_buffer_store_b8(b, gate, i, 0, 0); }
  __device__ void put_word(int32_t off, uint32_t w) const { __builtin_amdgcn_raw_buffer_store_b32(w, gate, off, 0, 0); }
};

// The gate producer of segment c.
__device__ inline GateRes gate_res(const GateArgs& a, const SelCtx& c) {
  GateRes p;
  gate_buffers(a, c, p.rho, p.gate);
  p.needs_class = true;
  p.aligned = (reinterpret_cast<uintptr_t>(a.gate + c.ubase + size_t(c.s0)) & 3u) == 0;
  return p;
}

// Work-group (sequence, unit): the whole segment's gate bytes and tau.
__global__ __launch_bounds__(kResThreads) void gate_resident_kernel(GateArgs a) {
  __shared__ ResShared sh;
  const Layout& lay = a.lay;
  SelCtx c;
  c.seq = blockIdx.x;
  c.s0 = lay.cu_seqlens[c.seq];
  c.n = lay.cu_seqlens[c.seq + 1] - c.s0;
  c.part = 0;
  c.ubase = size_t(blockIdx.y) * lay.total_tokens;
  SeqFrames<true> fr;
  fr.meta = lay.frame_meta;
  fr.fs = sh.fstart;
  fr.fe = sh.fend;
  fr.f0 = lay.cu_frames[c.seq];
  fr.nf = lay.cu_frames[c.seq + 1] - fr.f0;
  int32_t nh = 0;  // N_hist: every frame of the sequence but the last
  for (int32_t f = threadIdx.x; f < fr.nf; f += kResThreads) {
    const int32_t* m = lay.frame_meta + 3 * (fr.f0 + f);
    sh.fstart[f] = m[0];
    sh.fend[f] = m[0] + m[1] * m[2];
    if (f + 1 < fr.nf) nh += m[1] * m[2];
  }
  nh = wave_sum(nh);
  if ((threadIdx.x & 63) == 0) sh.wlt[threadIdx.x >> 6] = nh;
  __syncthreads();
  int32_t n_hist = 0;
  for (int w = 0; w < kResWaves; ++w) n_hist += sh.wlt[w];
  c.k = min(lay.cu_budget[c.seq + 1] - lay.cu_budget[c.seq], n_hist);
  __syncthreads();  // every thread has read the partial sums before the selection reuses them
  GateRes p;
  gate_buffers(a, c, p.rho, p.gate);
  p.needs_class = true;
  const uint32_t T = res_select(p, sh, fr, c);
  if (a.tau && threadIdx.x == 0)
    a.tau[size_t(blockIdx.y) * lay.n_seqs + c.seq] = c.k > 0 ? order_key_value(T) : __builtin_nanf("");
}

// Splitter path (segsel_split.h).  Work-group (1, seq, unit): k = min(B,
// N_hist) and the splitters of the segment.
template <bool LDS>
__global__ __launch_bounds__(kSpThreads) void gate_split_sample_kernel(GateArgs a) {
  __shared__ SpSampleShared sh;
  __shared__ int32_t nh_s;
  const Layout& lay = a.lay;
  SelCtx c = sel_ctx(lay);
  const int32_t budget = lay.cu_budget[c.seq + 1] - lay.cu_budget[c.seq];
  const GateRes p = gate_res(a, c);
  SpGather<GateRes> g;
  sp_gather(p, lay, c, g);  // the sample's loads first: the frame table's overlap them
  const SeqFrames<LDS> fr = sp_frames<LDS>(sh.fstart, sh.fend, lay, c.seq);
  if (LDS) __syncthreads();
  if (threadIdx.x < 64) {  // N_hist: every frame of the sequence but the last
    int32_t nh = 0;
    for (int32_t f = threadIdx.x; f + 1 < fr.nf; f += 64) nh += fr.end(f) - fr.start(f);
    nh = wave_sum(nh);
    if (threadIdx.x == 0) nh_s = nh;
  }
  __syncthreads();
  c.k = min(budget, nh_s);
  split_sample(p, sh, fr, a.sel, lay, c, nh_s, g);
}

// Work-group (part, seq, unit): the gate bytes the splitters decide.
__global__ __launch_bounds__(kSpPassThreads) void gate_split_classify_kernel(GateArgs a) {
  __shared__ SpPassShared sh;
  const SelCtx c = sel_ctx(a.lay);
  split_classify(gate_res(a, c), sh, a.sel, a.lay, c);
}

// Work-group (1, seq, unit): T, the open gate bytes and tau.
__global__ __launch_bounds__(kSpThreads) void gate_split_resolve_kernel(GateArgs a) {
  __shared__ SpResolveShared sh;
  const SelCtx c = sel_ctx(a.lay);
  int32_t mode;
  const uint32_t T = split_resolve<false>(gate_res(a, c), sh, a.sel, a.lay, c, &mode);
  if (a.tau && threadIdx.x == 0)
    a.tau[size_t(blockIdx.z) * a.lay.n_seqs + c.seq] = mode != kModeNone ? order_key_value(T) : __builtin_nanf("");
}

}  // namespace

hipError_t launch_gate_select(const GateArgs& g, hipStream_t stream) {
  switch (g.sel.path) {
    case kSelPathResident:
      if (g.lay.n_units == 0 || g.lay.n_seqs == 0) return hipSuccess;
      hipLaunchKernelGGL(gate_resident_kernel, dim3(g.lay.n_seqs, g.lay.n_units), dim3(kResThreads), 0, stream, g);
      return hipGetLastError();
    case kSelPathSplit:
      return launch_split(g.sel.lds_frames ? gate_split_sample_kernel<true> : gate_split_sample_kernel<false>,
                          gate_split_classify_kernel, gate_split_resolve_kernel,
                          static_cast<void (*)(GateArgs)>(nullptr), g, g.lay, stream);
    default:
      return launch_sel_passes(g.sel.lds_frames ? gate_produce_kernel<true> : gate_produce_kernel<false>,
                               gate_emit_kernel, g, g.sel, g.lay, stream);
  }
}

}  // namespace stlite
