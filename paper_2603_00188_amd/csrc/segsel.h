// Exact k-smallest selection over segments, spread over the whole GPU.
//
// A segment is one (unit, sequence) pair: the n tokens of one sequence in one
// (layer, kv head) unit.  Every token gets a 32-bit order key and the k keys
// first in (key ascending, index ascending) order are selected.  The TSG gate
// uses key = order_key(rho) on historical tokens and an all-ones key that is
// never selected on the others; the flat top-B uses key = ~order_key(S).
//
// Each segment is cut into P parts of whole 256-key groups (P from the host,
// the same for every segment) and every kernel runs one work-group of 512
// threads per (part, sequence, unit).  Inside a part each of the 8 waves owns a
// contiguous range.  Four kernels, one radix digit each (11, 11, 10 bits):
//   produce  the call computes the keys from its inputs and stores them; the
//            part's histogram of the top 11 bits goes to the workspace;
//   level 1  every work-group of the segment finds the level-0 pivot bin from
//            the parts' histograms (the same answer in each) and counts the
//            next 11 bits of its part's keys in that bin;
//   level 2  likewise for the last 10 bits of the keys matching the 22-bit
//            prefix, with the part's count of keys below that prefix;
//   emit     the level-2 pivot gives the exact k-th key T and need = how many
//            keys equal to T are taken; a part's output offset follows from
//            the earlier parts' level-2 histograms, a wave's from one counting
//            pass over its range; each wave then walks its range in index
//            order and ballots rank every taken key (keys equal to T taken
//            lowest index first).
// Each part histogram is stored fine and in 32-bin groups, so a pivot reads
// P x (groups + 32) counters instead of P x bins.  The key workspace is read
// back from L2 or the last-level cache.  There are no global atomics and no
// waits between work-groups.
#pragma once

#include "stlite_internal.h"
#include "tile_lds.h"

namespace stlite {

constexpr int kSelThreads = 512;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelJ = 8;              // tokens per lane per produce step (one 4-byte load each)
constexpr int kSelQ = 8;              // 16-byte key loads per lane per step of the key passes

constexpr uint32_t kSelNever = 0xffffffffu;  // key of a token that is never selected
// Largest key of a token that can be selected: below every key whose top 16
// bits are all ones, so that a 16-bit key prefix of 0xffff means "never"
// (only NaN scores map above it; they rank after every number, as one class).
constexpr uint32_t kSelKeyMax = 0xfffeffffu;

// Workspace words of one part histogram (fine bins, then the sums of 32-bin groups).
constexpr int kSelH0 = 2048 + 64;     // levels 0 and 1
constexpr int kSelH2 = 1024 + 32;     // level 2

// Part of a segment: keys [pa, pb) of n; the calling wave's range [lo, hi) inside it.
struct SelPart {
  int32_t pa, pb, lo, hi;
};

__device__ inline SelPart sel_part(int32_t n, int32_t parts, int32_t p) {
  SelPart r;
  const int32_t plen = ((n + parts * 256 - 1) / (parts * 256)) * 256;
  r.pa = min(p * plen, n);
  r.pb = min(r.pa + plen, n);
  const int32_t wlen = ((r.pb - r.pa + kSelWaves * 256 - 1) / (kSelWaves * 256)) * 256;
  // the wave's range is wave-uniform: keep it in scalar registers so that the
  // loops over it branch on scalars
  r.lo = __builtin_amdgcn_readfirstlane(min(r.pa + int32_t(threadIdx.x >> 6) * wlen, r.pb));
  r.hi = __builtin_amdgcn_readfirstlane(min(r.lo + wlen, r.pb));
  return r;
}

// Segment state words.
enum : int { kStK = 0, kStPrefix0, kStRem0, kStPrefix1, kStRem1, kStWords = 8 };

constexpr int kSelMaxParts = 16;

struct SelShared {
  uint32_t hist[2048];
  int32_t fstart[kSelFrames];
  int32_t fend[kSelFrames];
  int32_t red[kSelWaves];
  int32_t wlt[kSelWaves];
  int32_t weq[kSelWaves];
  int32_t wout[kSelWaves];
  int32_t weqb[kSelWaves];
  int32_t plt[kSelMaxParts];
  int32_t peq[kSelMaxParts];
  uint32_t gsum[64];
  uint32_t bsum[32];
  int32_t pg, pbefore, pbin, prem;
};

// The frames of one sequence, read from the LDS copy made by load_frames
// (LDS = true, at most kSelFrames frames) or from frame_meta.
template <bool LDS>
struct SeqFrames {
  const int32_t* meta;
  const int32_t* fs;  // LDS: first token of each frame
  const int32_t* fe;  // LDS: one past its last token
  int32_t f0, nf;

  __device__ int32_t start(int32_t f) const {
    if constexpr (LDS) return fs[f];
    else return meta[3 * (f0 + f)];
  }
  __device__ int32_t end(int32_t f) const {
    if constexpr (LDS) return fe[f];
    else return meta[3 * (f0 + f)] + meta[3 * (f0 + f) + 1] * meta[3 * (f0 + f) + 2];
  }
  // Last frame whose first token is <= tok, or -1.
  __device__ int32_t find(int32_t tok) const {
    int32_t lo = 0, hi = nf - 1, hit = -1;
    while (lo <= hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (start(mid) <= tok) { hit = mid; lo = mid + 1; } else { hi = mid - 1; }
    }
    return hit;
  }
};

enum TokClass : int { kText = 0, kHist = 1, kCurrent = 2 };

// The frames that overlap one wave step [base, base + span) of a sequence, as
// up to kStepFrames [start, end) ranges; n = -1 when more frames overlap it.
// Found from a cursor (last frame starting at or before the previous step's
// base) that only moves forward, with every lane reading the same addresses.
constexpr int kStepFrames = 4;
struct StepFrames {
  int32_t n;
  int32_t s[kStepFrames], e[kStepFrames];
  bool last[kStepFrames];  // the sequence's current (last) frame

  // Class shared by every token of [base, base + span), or -1 when the step
  // holds tokens of more than one class.
  __device__ int uniform(int32_t base, int32_t span) const {
    if (n == 0) return kText;
    if (n == 1 && s[0] <= base && e[0] >= base + span) return last[0] ? kCurrent : kHist;
    return -1;
  }

  __device__ int cls(int32_t tok) const {
    int c = kText;
#pragma unroll
    for (int q = 0; q < kStepFrames; ++q)
      if (q < n && tok >= s[q] && tok < e[q]) c = last[q] ? kCurrent : kHist;
    return c;
  }
};

// Every value here is wave-uniform (readfirstlane keeps it in scalar
// registers, so the loops branch on scalars).
template <bool LDS>
__device__ __forceinline__ StepFrames step_frames(const SeqFrames<LDS>& fr, int32_t& cur, int32_t base, int32_t span) {
  auto uni = [](int32_t x) { return __builtin_amdgcn_readfirstlane(x); };
  base = uni(base);
  cur = uni(cur);
  while (cur + 1 < fr.nf && uni(fr.start(cur + 1)) <= base) ++cur;
  StepFrames st;
  st.n = 0;
  int32_t f = (cur >= 0 && uni(fr.end(cur)) > base) ? cur : cur + 1;
  // static slots (no runtime index into the arrays, which would put them in
  // private memory)
#pragma unroll
  for (int q = 0; q < kStepFrames; ++q) {
    st.s[q] = 0;
    st.e[q] = 0;
    st.last[q] = false;
    if (f < fr.nf) {
      const int32_t s = uni(fr.start(f));
      if (s < base + span) {
        st.s[q] = s;
        st.e[q] = uni(fr.end(f));
        st.last[q] = f == fr.nf - 1;
        st.n = q + 1;
        ++f;
      }
    }
  }
  if (f < fr.nf && uni(fr.start(f)) < base + span) st.n = -1;  // more frames overlap the step
  return st;
}

// Class of token tok by a per-lane search (steps that overlap many frames).
template <bool LDS>
__device__ __forceinline__ int tok_class_search(const SeqFrames<LDS>& fr, int32_t tok) {
  const int32_t f = fr.find(tok);
  if (f < 0 || tok >= fr.end(f)) return kText;
  return f == fr.nf - 1 ? kCurrent : kHist;
}

// Frames of sequence seq; with LDS, copies their ranges into sh first (the
// caller synchronises before using them).
template <bool LDS>
__device__ inline SeqFrames<LDS> load_frames(SelShared& sh, const Layout& lay, int32_t seq) {
  SeqFrames<LDS> fr;
  fr.meta = lay.frame_meta;
  fr.fs = sh.fstart;
  fr.fe = sh.fend;
  fr.f0 = lay.cu_frames[seq];
  fr.nf = lay.cu_frames[seq + 1] - fr.f0;
  if constexpr (LDS) {
    for (int32_t f = threadIdx.x; f < fr.nf; f += kSelThreads) {
      const int32_t* m = lay.frame_meta + 3 * (fr.f0 + f);
      sh.fstart[f] = m[0];
      sh.fend[f] = m[0] + m[1] * m[2];
    }
  }
  return fr;
}

// hist[digit] += 1 for every lane with pred.  Up to ROUNDS digits shared by
// several lanes of the wave are aggregated first (leader lane, one LDS atomic
// each), so long runs of equal keys do not serialise on one LDS address; the
// remaining lanes add one by one.  Wave-uniform call.
template <int ROUNDS>
__device__ __forceinline__ void sel_hist_add(uint32_t* hist, bool pred, uint32_t digit) {
  const int lane = threadIdx.x & 63;
  uint64_t act = __ballot(pred);
#pragma unroll
  for (int round = 0; round < ROUNDS; ++round) {
    if (act == 0) return;
    const int leader = __ffsll((unsigned long long)act) - 1;
    const uint32_t ld = uint32_t(__builtin_amdgcn_readlane(int(digit), leader));
    const bool mine = pred && digit == ld;
    const uint64_t same = __ballot(mine);
    if (lane == leader) atomicAdd(&hist[ld], uint32_t(__popcll(same)));
    pred = pred && !mine;
    act &= ~same;
  }
  if (act != 0 && pred) atomicAdd(&hist[digit], 1u);
}

// hist[digit] += 1 for every lane with pred, for sparse predicates with spread
// digits: one atomic per lane, except that a wave whose active lanes all share
// one digit adds them with one atomic.  Wave-uniform call.
__device__ __forceinline__ void sel_hist_add_sparse(uint32_t* hist, bool pred, uint32_t digit) {
  const uint64_t act = __ballot(pred);
  if (act == 0) return;
  const int leader = __ffsll((unsigned long long)act) - 1;
  const uint32_t ld = uint32_t(__builtin_amdgcn_readlane(int(digit), leader));
  if (__ballot(pred && digit != ld) == 0) {
    if (int(threadIdx.x & 63) == leader) atomicAdd(&hist[ld], uint32_t(__popcll(act)));
  } else if (pred) {
    atomicAdd(&hist[digit], 1u);
  }
}

__device__ __forceinline__ int32_t wave_sum(int32_t x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Inclusive scan over the wave.
__device__ __forceinline__ int32_t wave_inscan(int32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

// Exclusive scan over the wave of x in [0, 7]; *total gets the wave's sum.
__device__ __forceinline__ int32_t wave_exscan7(int32_t x, int32_t* total) {
  const uint64_t below = (uint64_t(1) << (threadIdx.x & 63)) - 1;
  const uint64_t b0 = __ballot(x & 1), b1 = __ballot(x & 2), b2 = __ballot(x & 4);
  *total = __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2);
  return __popcll(b0 & below) + 2 * __popcll(b1 & below) + 4 * __popcll(b2 & below);
}

// Zero the first nb words of sh.hist.  The caller synchronises.
__device__ __forceinline__ void sel_hist_zero(SelShared& sh, int nb) {
  for (int b = threadIdx.x; b < nb; b += kSelThreads) sh.hist[b] = 0;
}

// Store sh.hist (NB fine bins) as one part histogram: the fine bins, then the
// sums of each group of 32.  The caller has synchronised after the counting.
template <int NB>
__device__ __forceinline__ void sel_hist_store(const SelShared& sh, uint32_t* dst) {
  for (int b = threadIdx.x; b < NB; b += kSelThreads) dst[b] = sh.hist[b];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int g = wave; g < NB / 32; g += kSelWaves) {  // one group per wave, in its low 32 lanes
    uint32_t v = lane < 32 ? sh.hist[g * 32 + lane] : 0u;
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) dst[NB + g] = v;
  }
}

// Pivot of one level from the parts' histograms (part stride `stride` words,
// NB fine bins then NB / 32 group sums): the bin holding rank k_rem of the
// keys counted, and the rank inside it.  Every thread calls it; the parts'
// counters are loaded by the whole work-group at once and summed with LDS
// atomics, first the group sums, then the 32 bins of the chosen group.
template <int NB>
__device__ __forceinline__ void sel_pivot_parts(SelShared& sh, const uint32_t* h, int32_t stride, int32_t parts,
                                                int32_t k_rem, int32_t* bin_out, int32_t* rem_out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int NG = NB / 32;
  if (threadIdx.x < 64) sh.gsum[threadIdx.x] = 0u;
  if (threadIdx.x < 32) sh.bsum[threadIdx.x] = 0u;
  __syncthreads();
  for (int32_t i = threadIdx.x; i < parts * NG; i += kSelThreads) {
    const uint32_t v = h[size_t(i / NG) * stride + NB + i % NG];
    if (v) atomicAdd(&sh.gsum[i % NG], v);
  }
  __syncthreads();
  if (wave == 0) {
    const int32_t c = lane < NG ? int32_t(sh.gsum[lane]) : 0;
    const int32_t incl = wave_inscan(c);
    const uint64_t m = __ballot(lane < NG && incl >= k_rem);  // first group whose running count reaches k_rem
    const int g = m ? __ffsll((unsigned long long)m) - 1 : NG - 1;
    if (lane == g) {
      sh.pg = g;
      sh.pbefore = incl - c;
    }
  }
  __syncthreads();
  const int g = sh.pg;
  for (int32_t i = threadIdx.x; i < parts * 32; i += kSelThreads) {
    const uint32_t v = h[size_t(i / 32) * stride + g * 32 + i % 32];
    if (v) atomicAdd(&sh.bsum[i % 32], v);
  }
  __syncthreads();
  if (wave == 0) {
    const int32_t f = lane < 32 ? int32_t(sh.bsum[lane]) : 0;
    const int32_t fin = wave_inscan(f) + sh.pbefore;
    const uint64_t m2 = __ballot(lane < 32 && fin >= k_rem);
    const int b = m2 ? __ffsll((unsigned long long)m2) - 1 : 31;
    if (lane == b) {
      sh.pbin = g * 32 + b;
      sh.prem = k_rem - (fin - f);
    }
  }
  __syncthreads();
  *bin_out = sh.pbin;
  *rem_out = sh.prem;
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Four keys of the lane at segment index i (a multiple of 4) through the
// segment's key buffer; keys at or past hi read as kSelNever.
__device__ __forceinline__ uint4 sel_load4(__amdgpu_buffer_rsrc_t r, int32_t i, int32_t hi) {
  const u32x4_t w = __builtin_amdgcn_raw_buffer_load_b128(r, i * 4, 0, 0);
  return make_uint4(i < hi ? w.x : kSelNever, i + 1 < hi ? w.y : kSelNever, i + 2 < hi ? w.z : kSelNever,
                    i + 3 < hi ? w.w : kSelNever);
}

// Per-segment context handed to the call's producer and consumer.
struct SelCtx {
  int32_t seq, s0, n;  // sequence, its first token, its length
  int32_t k;           // keys to select
  int32_t part;        // blockIdx.x
  size_t ubase;        // unit * total_tokens
};

// Grid of every selection kernel: (part, sequence, unit).
__device__ inline size_t sel_seg(const Layout& lay) { return size_t(blockIdx.z) * lay.n_seqs + blockIdx.y; }

__device__ inline SelCtx sel_ctx(const Layout& lay) {
  SelCtx c;
  c.seq = blockIdx.y;
  c.s0 = lay.cu_seqlens[c.seq];
  c.n = lay.cu_seqlens[c.seq + 1] - c.s0;
  c.k = 0;
  c.part = blockIdx.x;
  c.ubase = size_t(blockIdx.z) * lay.total_tokens;
  return c;
}

// The segment's keys as a raw buffer over its whole 16-byte groups (the key
// row is padded for them); offsets past the end read 0 and drop stores.
__device__ inline __amdgpu_buffer_rsrc_t sel_keys(const SelPlan& s, const Layout& lay, const SelCtx& c) {
  uint32_t* base = s.keys + size_t(blockIdx.z) * sel_key_stride(lay.total_tokens, lay.n_seqs) + sel_key_base(c.s0, c.seq);
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, ((c.n + 3) / 4) * 16, kBufferFlags);
}

// Produce pass: keys of this part and its level-0 histogram.  Prod provides
//   int32_t cursor(const SelCtx&, int32_t i): wave-uniform frame cursor for segment token i;
//   Raw: the loaded inputs of one step;
//   void fetch(const SelCtx&, int32_t base, int32_t lane, int32_t& cur, Raw&): issue the
//        loads of segment tokens base + 64 j + lane (and classify them);
//   void finish(const SelCtx&, int32_t base, int32_t lane, int32_t hi, const Raw&, uint32_t (&key)[kSelJ]):
//        their keys, kSelNever where base + 64 j + lane >= hi.
// The loads of step s + 1 are issued before step s is finished, so a wave
// keeps one step's loads in flight while it computes.  c.k is written to the
// segment state by part 0.
template <class Prod>
__device__ void sel_produce(const Prod& p, SelShared& sh, const SelPlan& s, const Layout& lay, const SelCtx& c) {
  const int lane = threadIdx.x & 63;
  const SelPart pt = sel_part(c.n, s.parts, c.part);
  const __amdgpu_buffer_rsrc_t keys = sel_keys(s, lay, c);
  const int32_t dropped = ((c.n + 3) / 4) * 16;  // a store offset the buffer drops
  sel_hist_zero(sh, 2048);
  __syncthreads();
  int32_t cur = p.cursor(c, pt.lo);
  // (a fetch past the part reads inside the sequence or gets 0 from the
  // buffer, and its result is never finished)
  typename Prod::Raw raw;
  p.fetch(c, pt.lo, lane, cur, raw);
  for (int32_t base = pt.lo; base < pt.hi; base += 64 * kSelJ) {
    typename Prod::Raw next;
    p.fetch(c, base + 64 * kSelJ, lane, cur, next);
    uint32_t key[kSelJ];
    p.finish(c, base, lane, pt.hi, raw, key);
#pragma unroll
    for (int j = 0; j < kSelJ; ++j) {
      const int32_t i = base + 64 * j + lane;
      __builtin_amdgcn_raw_buffer_store_b32(key[j], keys, i < pt.hi ? i * 4 : dropped, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kSelJ; ++j) sel_hist_add<1>(sh.hist, base + 64 * j + lane < pt.hi, key[j] >> 21);
    raw = next;
  }
  __syncthreads();
  const size_t seg = sel_seg(lay);
  sel_hist_store<2048>(sh, s.hist0 + (seg * s.parts + c.part) * kSelH0);
  if (c.part == 0 && threadIdx.x == 0) s.state[seg * kStWords + kStK] = c.k;
}

// Level 1: pivot of level 0, then the part's histogram of bits 20..10 of the
// keys in the pivot bin.
__device__ inline void sel_level1(SelShared& sh, const SelPlan& s, const Layout& lay, const SelCtx& c) {
  const int lane = threadIdx.x & 63;
  const size_t seg = sel_seg(lay);
  int32_t* st = s.state + seg * kStWords;
  const int32_t k = st[kStK];
  if (k <= 0) return;
  int32_t bin, rem;
  sel_pivot_parts<2048>(sh, s.hist0 + seg * s.parts * kSelH0, kSelH0, s.parts, k, &bin, &rem);
  if (c.part == 0 && threadIdx.x == 0) {
    st[kStPrefix0] = int32_t(uint32_t(bin) << 21);
    st[kStRem0] = rem;
  }
  sel_hist_zero(sh, 2048);
  __syncthreads();
  const uint32_t p0 = uint32_t(bin);
  const SelPart pt = sel_part(c.n, s.parts, c.part);
  const __amdgpu_buffer_rsrc_t keys = sel_keys(s, lay, c);
  for (int32_t base = pt.lo; base < pt.hi; base += 256 * kSelQ) {
    uint4 v[kSelQ];
#pragma unroll
    for (int q = 0; q < kSelQ; ++q) v[q] = sel_load4(keys, base + 256 * q + 4 * lane, pt.hi);
#pragma unroll
    for (int q = 0; q < kSelQ; ++q) {
      const uint32_t kk[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
      for (int e = 0; e < 4; ++e)  // padding reads as kSelNever, which no selected key equals
        sel_hist_add_sparse(sh.hist, kk[e] != kSelNever && (kk[e] >> 21) == p0, (kk[e] >> 10) & 2047u);
    }
  }
  __syncthreads();
  sel_hist_store<2048>(sh, s.hist1 + (seg * s.parts + c.part) * kSelH0);
}

// Level 2: pivot of level 1, then the part's histogram of bits 9..0 of the
// keys matching the 22-bit prefix and its count of keys below that prefix.
__device__ inline void sel_level2(SelShared& sh, const SelPlan& s, const Layout& lay, const SelCtx& c) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t seg = sel_seg(lay);
  int32_t* st = s.state + seg * kStWords;
  const int32_t k = st[kStK];
  if (k <= 0) return;
  const uint32_t pre0 = uint32_t(st[kStPrefix0]);
  int32_t bin, rem;
  sel_pivot_parts<2048>(sh, s.hist1 + seg * s.parts * kSelH0, kSelH0, s.parts, st[kStRem0], &bin, &rem);
  const uint32_t p22 = pre0 | (uint32_t(bin) << 10);
  if (c.part == 0 && threadIdx.x == 0) {
    st[kStPrefix1] = int32_t(p22);
    st[kStRem1] = rem;
  }
  sel_hist_zero(sh, 1024);
  __syncthreads();
  const SelPart pt = sel_part(c.n, s.parts, c.part);
  const __amdgpu_buffer_rsrc_t keys = sel_keys(s, lay, c);
  int32_t below = 0;
  for (int32_t base = pt.lo; base < pt.hi; base += 256 * kSelQ) {
    uint4 v[kSelQ];
#pragma unroll
    for (int q = 0; q < kSelQ; ++q) v[q] = sel_load4(keys, base + 256 * q + 4 * lane, pt.hi);
#pragma unroll
    for (int q = 0; q < kSelQ; ++q) {
      const uint32_t kk[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        below += kk[e] < p22 ? 1 : 0;
        sel_hist_add_sparse(sh.hist, kk[e] != kSelNever && (kk[e] >> 10) == (p22 >> 10), kk[e] & 1023u);
      }
    }
  }
  below = wave_sum(below);
  if (lane == 0) sh.red[wave] = below;
  __syncthreads();
  sel_hist_store<1024>(sh, s.hist2 + (seg * s.parts + c.part) * kSelH2);
  if (threadIdx.x == 0) {
    int32_t t = 0;
    for (int w = 0; w < kSelWaves; ++w) t += sh.red[w];
    s.below[seg * s.parts + c.part] = t;
  }
}

// Emit pass.  Prod provides
//   void emit(const SelCtx&, int32_t i, uint32_t key, bool take, int32_t pos):
//        called for every token i of the part, with take (selected) and pos
//        (its rank among the segment's selected keys, when taken).
// Sets c.k; returns T (the k-th key) when c.k > 0.
template <class Prod>
__device__ uint32_t sel_emit(const Prod& p, SelShared& sh, const SelPlan& s, const Layout& lay, SelCtx& c) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t seg = sel_seg(lay);
  const int32_t* st = s.state + seg * kStWords;
  const int32_t k = st[kStK];
  c.k = k;
  const SelPart pt = sel_part(c.n, s.parts, c.part);
  const __amdgpu_buffer_rsrc_t keys = sel_keys(s, lay, c);
  uint32_t T = 0u;
  int32_t need = 0;
  if (k > 0) {
    const uint32_t* h2 = s.hist2 + seg * s.parts * kSelH2;
    int32_t bin, rem;
    sel_pivot_parts<1024>(sh, h2, kSelH2, s.parts, st[kStRem1], &bin, &rem);
    T = uint32_t(st[kStPrefix1]) | uint32_t(bin);
    need = rem;
    // keys < T and == T in each earlier part: its count below the 22-bit
    // prefix, its level-2 groups below T's group and the bins of T's group
    // below T (64 counters per part, loaded by the whole work-group at once)
    const uint32_t tl = T & 1023u;
    if (threadIdx.x < kSelMaxParts) sh.plt[threadIdx.x] = 0;
    __syncthreads();
    for (int32_t i = threadIdx.x; i < c.part * 64; i += kSelThreads) {
      const int32_t q = i / 64, j = i % 64;
      const uint32_t* h = h2 + size_t(q) * kSelH2;
      int32_t v = 0;
      if (j < 32) {
        if (uint32_t(j) < (tl >> 5)) v = int32_t(h[1024 + j]);
      } else if (uint32_t(j - 32) < (tl & 31u)) {
        v = int32_t(h[(tl & ~31u) + uint32_t(j - 32)]);
      }
      if (j == 0) {
        v += s.below[seg * s.parts + q];
        sh.peq[q] = int32_t(h[tl]);
      }
      if (v) atomicAdd(&sh.plt[q], v);
    }
    // keys < T and == T in each wave's range of this part
    int32_t lt = 0, eq = 0;
    for (int32_t base = pt.lo; base < pt.hi; base += 256 * kSelQ) {
      uint4 v[kSelQ];
#pragma unroll
      for (int q = 0; q < kSelQ; ++q) v[q] = sel_load4(keys, base + 256 * q + 4 * lane, pt.hi);
#pragma unroll
      for (int q = 0; q < kSelQ; ++q) {
        const uint32_t kk[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {  // padding (kSelNever) is never < T or == T
          lt += kk[e] < T ? 1 : 0;
          eq += kk[e] == T ? 1 : 0;
        }
      }
    }
    lt = wave_sum(lt);
    eq = wave_sum(eq);
    if (lane == 0) {
      sh.wlt[wave] = lt;
      sh.weq[wave] = eq;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t out = 0, eq_before = 0;
      for (int32_t q = 0; q < c.part; ++q) {
        out += sh.plt[q] + min(max(need - eq_before, 0), sh.peq[q]);
        eq_before += sh.peq[q];
      }
      for (int w = 0; w < kSelWaves; ++w) {
        sh.wout[w] = out;
        sh.weqb[w] = eq_before;
        out += sh.wlt[w] + min(max(need - eq_before, 0), sh.weq[w]);
        eq_before += sh.weq[w];
      }
    }
    __syncthreads();
  }
  int32_t out = k > 0 ? sh.wout[wave] : 0;
  int32_t eq_rank = k > 0 ? sh.weqb[wave] : 0;
  for (int32_t base = pt.lo; base < pt.hi; base += 256 * kSelQ) {
    uint4 v[kSelQ];
#pragma unroll
    for (int q = 0; q < kSelQ; ++q) v[q] = sel_load4(keys, base + 256 * q + 4 * lane, pt.hi);
#pragma unroll
    for (int q = 0; q < kSelQ; ++q) {
      const int32_t i0 = base + 256 * q + 4 * lane;
      const uint32_t kk[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
      bool less[4], eq[4];
      int32_t n_eq = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool in = i0 + e < pt.hi;
        less[e] = k > 0 && in && kk[e] < T;
        eq[e] = k > 0 && in && kk[e] == T;
        n_eq += eq[e] ? 1 : 0;
      }
      int32_t eq_tot;
      int32_t r = eq_rank + wave_exscan7(n_eq, &eq_tot);
      bool take[4];
      int32_t n_take = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        take[e] = less[e] || (eq[e] && r < need);
        r += eq[e] ? 1 : 0;
        n_take += take[e] ? 1 : 0;
      }
      int32_t take_tot;
      int32_t pos = out + wave_exscan7(n_take, &take_tot);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (i0 + e < pt.hi) p.emit(c, i0 + e, kk[e], take[e], pos);
        pos += take[e] ? 1 : 0;
      }
      out += take_tot;
      eq_rank += eq_tot;
    }
  }
  return T;
}

namespace {

__global__ __launch_bounds__(kSelThreads) void sel_level1_kernel(SelPlan s, Layout lay) {
  __shared__ SelShared sh;
  sel_level1(sh, s, lay, sel_ctx(lay));
}

__global__ __launch_bounds__(kSelThreads) void sel_level2_kernel(SelPlan s, Layout lay) {
  __shared__ SelShared sh;
  sel_level2(sh, s, lay, sel_ctx(lay));
}

}  // namespace

// The four passes over grid (parts, sequences, units).
template <class Args>
hipError_t launch_sel_passes(void (*produce)(Args), void (*emit)(Args), const Args& a, const SelPlan& s,
                             const Layout& lay, hipStream_t stream) {
  if (lay.n_units == 0) return hipSuccess;
  const dim3 grid(s.parts, lay.n_seqs, lay.n_units);
  hipLaunchKernelGGL(produce, grid, dim3(kSelThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sel_level1_kernel, grid, dim3(kSelThreads), 0, stream, s, lay);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sel_level2_kernel, grid, dim3(kSelThreads), 0, stream, s, lay);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(emit, grid, dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
