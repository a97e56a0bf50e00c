// Integrated score and flat top-B (Eq. modal_scoring and Sec. integrated
// scoring of the paper), for every (unit, sequence) segment at once:
//   S = A on text tokens, S = M * (A + alpha * Phi) on visual tokens,
//   I_keep = the B tokens first in (S descending, index ascending) order,
//   written in ascending token order.
// The selection is the per-segment radix select of segsel.h on the keys
// ~order_key(S) (ascending key = descending S).
#include "segsel.h"
#include "segsel_resident.h"
#include "segsel_split.h"
#include "stlite_internal.h"

namespace stlite {
namespace {

template <bool LDS>
struct SelectProd {
  __amdgpu_buffer_rsrc_t a_base;  // the segment's A, Phi and gate (out-of-range lanes read 0)
  __amdgpu_buffer_rsrc_t phi;
  __amdgpu_buffer_rsrc_t gate;
  bool has_phi, has_gate;
  float* score;          // nullable: the segment's S
  int32_t* kept;         // the segment's kept list
  float alpha;
  SeqFrames<LDS> fr;
  bool classify;  // Phi or the gate is given: visual tokens must be told from text

  __device__ int32_t cursor(const SelCtx& c, int32_t i) const {
    return classify ? __builtin_amdgcn_readfirstlane(fr.find(c.s0 + i)) : -1;
  }

  struct Raw {
    uint32_t vis;  // bit j: token j of the step is visual
    float A[kSelJ], ph[kSelJ];
    uint32_t g[kSelJ];
  };

  __device__ void fetch(const SelCtx& c, int32_t base, int32_t lane, int32_t& cur, Raw& r) const {
    r.vis = 0u;
    if (classify) {
      const StepFrames st = step_frames(fr, cur, c.s0 + base, 64 * kSelJ);
      const int u = st.n >= 0 ? st.uniform(c.s0 + base, 64 * kSelJ) : -1;
      if (u >= 0) {
        r.vis = u != kText ? (1u << kSelJ) - 1u : 0u;
      } else if (st.n >= 0) {
#pragma unroll
        for (int j = 0; j < kSelJ; ++j) r.vis |= (st.cls(c.s0 + base + 64 * j + lane) != kText ? 1u : 0u) << j;
      } else {
#pragma unroll
        for (int j = 0; j < kSelJ; ++j) r.vis |= (tok_class_search(fr, c.s0 + base + 64 * j + lane) != kText ? 1u : 0u) << j;
      }
    }
#pragma unroll
    for (int j = 0; j < kSelJ; ++j) {
      const int32_t i = base + 64 * j + lane;
      r.A[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(a_base, i * 4, 0, 0));
      r.ph[j] = has_phi ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(phi, i * 4, 0, 0)) : 0.0f;
      r.g[j] = has_gate ? __builtin_amdgcn_raw_buffer_load_b8(gate, i, 0, 0) : 1u;
    }
  }

  __device__ void finish(const SelCtx&, int32_t base, int32_t lane, int32_t hi, const Raw& r,
                         uint32_t (&key)[kSelJ]) const {
#pragma unroll
    for (int j = 0; j < kSelJ; ++j) {
      const int32_t i = base + 64 * j + lane;
      float S = r.A[j];
      if ((r.vis >> j) & 1u) {
        const float x = has_phi ? fmaf(alpha, r.ph[j], r.A[j]) : r.A[j];
        S = r.g[j] == 0 ? 0.0f : x;
      }
      if (score && i < hi) score[i] = S;
      key[j] = i < hi ? min(~order_key(S), kSelKeyMax) : kSelNever;
    }
  }

  __device__ void emit(const SelCtx& c, int32_t i, uint32_t, bool take, int32_t pos) const {
    if (take && pos < c.k) kept[pos] = c.s0 + i;
  }
};

template <bool LDS>
__device__ inline SelectProd<LDS> select_prod(const SelectArgs& a, const SelCtx& c) {
  SelectProd<LDS> p{};
  const size_t seg0 = c.ubase + size_t(c.s0);
  const int32_t n = c.n;
  p.a_base = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.a_base) + seg0, 0, n * 4, kBufferFlags);
  p.has_phi = a.phi != nullptr;
  p.has_gate = a.gate != nullptr;
  p.phi = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.has_phi ? a.phi + seg0 : a.a_base), 0, n * 4, kBufferFlags);
  p.gate = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.has_gate ? a.gate + seg0 : nullptr), 0,
                                             p.has_gate ? n : 0, kBufferFlags);
  p.score = a.score ? a.score + seg0 : nullptr;
  p.kept = a.kept + size_t(blockIdx.z) * a.lay.total_budget + a.lay.cu_budget[c.seq];
  p.alpha = a.alpha;
  return p;
}

// Work-group (part, seq, unit): scores and keys of one part of a segment.
// LDS: every sequence has at most kSelFrames frames (their ranges go to LDS).
template <bool LDS>
__global__ __launch_bounds__(kSelThreads) void select_produce_kernel(SelectArgs a) {
  __shared__ SelShared sh;
  SelCtx c = sel_ctx(a.lay);
  c.k = a.lay.cu_budget[c.seq + 1] - a.lay.cu_budget[c.seq];
  SelectProd<LDS> p = select_prod<LDS>(a, c);
  p.classify = a.phi != nullptr || a.gate != nullptr;
  p.fr = load_frames<LDS>(sh, a.lay, c.seq);
  __syncthreads();
  sel_produce(p, sh, a.sel, a.lay, c);
}

// Work-group (part, seq, unit): kept indices of one part of a segment.
__global__ __launch_bounds__(kSelThreads) void select_emit_kernel(SelectArgs a) {
  __shared__ SelShared sh;
  SelCtx c = sel_ctx(a.lay);
  const SelectProd<false> p = select_prod<false>(a, c);  // the emit pass reads keys only
  sel_emit(p, sh, a.sel, a.lay, c);
}

// The top-B of one segment held by one work-group (segsel_resident.h).
struct SelectRes {
  static constexpr int kGroup = 1;        // tiles a classifying wave loads at once (segsel_split.h)
  static constexpr bool kDirect = false;  // a ranked list: the splitter path emits it from codes
  static constexpr bool aligned = false;
  // The segment's A, Phi and gate (out-of-range lanes read 0).  A Phi or gate
  // the call does not give is a buffer of no records: its loads return 0
  // without touching memory, so every load is issued unconditionally.
  __amdgpu_buffer_rsrc_t a_base;
  __amdgpu_buffer_rsrc_t phi;
  __amdgpu_buffer_rsrc_t gate;
  bool has_phi, has_gate;
  uint32_t closed;   // the gate byte of a gated-out token: 0, or 256 (no byte) without a gate
  bool needs_class;  // Phi or the gate is given: visual tokens must be told from text
  float alpha;
  float* score;      // nullable: the segment's S
  int32_t* kept;     // the segment's kept list
  int32_t k, s0;

  struct Raw {
    float A[4], ph[4];
    uint32_t g[4];
  };

  __device__ void load(int32_t base, Raw& r) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int32_t i = base + 64 * e + lane;
      r.A[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(a_base, i * 4, 0, 0));
      r.ph[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(phi, i * 4, 0, 0));
      r.g[e] = __builtin_amdgcn_raw_buffer_load_b8(gate, i, 0, 0);
    }
  }

  // S of Eq. modal_scoring, as the four-pass producer computes it.
  __device__ float score_of(float A, float ph, uint32_t g, bool visual) const {
    if (!visual) return A;
    const float x = has_phi ? fmaf(alpha, ph, A) : A;
    return g == closed ? 0.0f : x;
  }

  __device__ void keys(int32_t base, const int (&cls)[4], int32_t hi, const Raw& r, uint32_t (&key)[4]) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int32_t i = base + 64 * e + lane;
      const float S = score_of(r.A[e], r.ph[e], r.g[e], cls[e] != kText);
      if (score && i < hi) score[i] = S;
      key[e] = i < hi ? min(~order_key(S), kSelKeyMax) : kSelNever;
    }
  }

  __device__ void emit(int32_t i, int, bool take, int32_t pos) const {
    if (take && pos < k) kept[pos] = s0 + i;
  }

  // Whether a token of class cls can be selected (segsel_split.h): all can.
  __device__ bool selectable(int) const { return true; }

  // keys() for a whole tile of one class (cls, wave-uniform) inside the segment.
  __device__ void keys_uniform(int32_t base, int cls, const Raw& r, uint32_t (&key)[4]) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float S = score_of(r.A[e], r.ph[e], r.g[e], cls != kText);
      if (score) score[base + 64 * e + lane] = S;
      key[e] = min(~order_key(S), kSelKeyMax);
    }
  }

  // The splitter path (segsel_split.h): one token's inputs and key, and a
  // taken token's kept entry at its rank.
  struct Raw1 {
    float A, ph;
    uint32_t g;
  };

  // The gate byte first; A and Phi only where S depends on them (a text
  // token, or a visual one whose gate is not zero).
  __device__ void load1(int32_t i, Raw1& r) const {
    r.g = __builtin_amdgcn_raw_buffer_load_b8(gate, i, 0, 0);
  }

  __device__ void load1_rest(int32_t i, int cls, Raw1& r) const {
    r.A = 0.0f;
    r.ph = 0.0f;
    if (cls == kText || r.g != closed) {
      r.A = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(a_base, i * 4, 0, 0));
      r.ph = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(phi, i * 4, 0, 0));
    }
  }

  __device__ uint32_t key1(const Raw1& r, int cls) const {
    return min(~order_key(score_of(r.A, r.ph, r.g, cls != kText)), kSelKeyMax);
  }

  __device__ void emit_code(int32_t i, bool, bool take, int32_t pos) const {
    if (take && pos < k) kept[pos] = s0 + i;
  }

  __device__ void put_byte(int32_t, uint8_t) const {}  // (kDirect only)
  __device__ void put_word(int32_t, uint32_t) const {}
};

// The producer of segment c of `unit` (score: write S, when the call asks for it).
__device__ inline SelectRes select_res(const SelectArgs& a, const SelCtx& c, int32_t unit, bool score) {
  SelectRes p;
  const size_t seg0 = c.ubase + size_t(c.s0);
  p.a_base = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.a_base) + seg0, 0, c.n * 4, kBufferFlags);
  p.has_phi = a.phi != nullptr;
  p.has_gate = a.gate != nullptr;
  p.phi = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.has_phi ? a.phi + seg0 : a.a_base), 0,
                                            p.has_phi ? c.n * 4 : 0, kBufferFlags);
  p.gate = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.has_gate ? a.gate + seg0 : nullptr), 0,
                                             p.has_gate ? c.n : 0, kBufferFlags);
  p.closed = p.has_gate ? 0u : 256u;
  p.needs_class = p.has_phi || p.has_gate;
  p.alpha = a.alpha;
  p.score = (score && a.score) ? a.score + seg0 : nullptr;
  p.kept = a.kept + size_t(unit) * a.lay.total_budget + a.lay.cu_budget[c.seq];
  p.k = c.k;
  p.s0 = c.s0;
  return p;
}

// Work-group (sequence, unit): the whole segment's kept list (and S).
__global__ __launch_bounds__(kResThreads) void select_resident_kernel(SelectArgs a) {
  __shared__ ResShared sh;
  const Layout& lay = a.lay;
  SelCtx c;
  c.seq = blockIdx.x;
  c.s0 = lay.cu_seqlens[c.seq];
  c.n = lay.cu_seqlens[c.seq + 1] - c.s0;
  c.part = 0;
  c.ubase = size_t(blockIdx.y) * lay.total_tokens;
  c.k = lay.cu_budget[c.seq + 1] - lay.cu_budget[c.seq];
  const SelectRes p = select_res(a, c, blockIdx.y, true);
  SeqFrames<true> fr;
  fr.meta = lay.frame_meta;
  fr.fs = sh.fstart;
  fr.fe = sh.fend;
  fr.f0 = lay.cu_frames[c.seq];
  fr.nf = lay.cu_frames[c.seq + 1] - fr.f0;
  for (int32_t f = threadIdx.x; f < fr.nf; f += kResThreads) {
    const int32_t* m = lay.frame_meta + 3 * (fr.f0 + f);
    sh.fstart[f] = m[0];
    sh.fend[f] = m[0] + m[1] * m[2];
  }
  __syncthreads();
  res_select(p, sh, fr, c);
}

// Splitter path (segsel_split.h), grids (1 or parts, seq, unit); k = B of the
// sequence.
template <bool LDS>
__global__ __launch_bounds__(kSpThreads) void select_split_sample_kernel(SelectArgs a) {
  __shared__ SpSampleShared sh;
  SelCtx c = sel_ctx(a.lay);
  c.k = a.lay.cu_budget[c.seq + 1] - a.lay.cu_budget[c.seq];
  const SelectRes p = select_res(a, c, blockIdx.z, false);
  SpGather<SelectRes> g;
  sp_gather(p, a.lay, c, g);  // the sample's loads first: the frame table's overlap them
  const SeqFrames<LDS> fr = sp_frames<LDS>(sh.fstart, sh.fend, a.lay, c.seq);
  __syncthreads();
  split_sample(p, sh, fr, a.sel, a.lay, c, c.n, g);
}

__global__ __launch_bounds__(kSpPassThreads) void select_split_classify_kernel(SelectArgs a) {
  __shared__ SpPassShared sh;
  SelCtx c = sel_ctx(a.lay);
  c.k = a.lay.cu_budget[c.seq + 1] - a.lay.cu_budget[c.seq];
  split_classify(select_res(a, c, blockIdx.z, true), sh, a.sel, a.lay, c);
}

__global__ __launch_bounds__(kSpThreads) void select_split_resolve_kernel(SelectArgs a) {
  __shared__ SpResolveShared sh;
  SelCtx c = sel_ctx(a.lay);
  c.k = a.lay.cu_budget[c.seq + 1] - a.lay.cu_budget[c.seq];
  int32_t mode;
  split_resolve<true>(select_res(a, c, blockIdx.z, false), sh, a.sel, a.lay, c, &mode);
}

__global__ __launch_bounds__(kSpPassThreads) void select_split_emit_kernel(SelectArgs a) {
  SelCtx c = sel_ctx(a.lay);
  c.k = a.lay.cu_budget[c.seq + 1] - a.lay.cu_budget[c.seq];
  split_emit(select_res(a, c, blockIdx.z, false), a.sel, a.lay, c);
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  switch (a.sel.path) {
    case kSelPathResident:
      if (a.lay.n_units == 0 || a.lay.n_seqs == 0) return hipSuccess;
      hipLaunchKernelGGL(select_resident_kernel, dim3(a.lay.n_seqs, a.lay.n_units), dim3(kResThreads), 0, stream, a);
      return hipGetLastError();
    case kSelPathSplit:
      return launch_split(a.sel.lds_frames ? select_split_sample_kernel<true> : select_split_sample_kernel<false>,
                          select_split_classify_kernel, select_split_resolve_kernel, select_split_emit_kernel, a,
                          a.lay, stream);
    default:
      return launch_sel_passes(a.sel.lds_frames ? select_produce_kernel<true> : select_produce_kernel<false>,
                               select_emit_kernel, a, a.sel, a.lay, stream);
  }
}

}  // namespace stlite
