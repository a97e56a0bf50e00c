// Exact k-smallest selection of a whole (unit, sequence) segment by one
// work-group, for segments of at most kResCapacity tokens (longer sequences
// take the four-pass selection of segsel.h).
//
// Same order and result as segsel.h: 32-bit order keys, the k keys first in
// (key ascending, index ascending) order.  One launch instead of four, the
// inputs read once and no key written to memory:
//   1. every wave walks its contiguous range of the segment in steps of 256
//      tokens (four rows of 64 consecutive tokens, one token per lane and
//      row), computes the keys, keeps them in registers and counts their top
//      11 bits in an LDS histogram;
//   2. two more walks over the keys in registers count the next 11 and the
//      last 10 bits of the keys that match the prefix found so far, which
//      gives the exact k-th key T and `need`, how many keys equal to T are
//      taken (lowest index first);
//   3. each wave counts its keys below and equal to T, the counts are scanned
//      over the waves, and each wave walks its range again in index order,
//      ranking the taken keys with ballots.
// The bound on a wave's steps keeps the fully unrolled walks (every register
// index static) short: measured against the four passes, one work-group per
// segment wins while a segment is a few tens of thousands of tokens long and
// the four launches dominate, and loses beyond, where the chip's 256 CUs
// stream the passes faster than one CU per segment.
#pragma once

#include "segsel.h"

namespace stlite {

constexpr int kResThreads = 1024;
constexpr int kResWaves = kResThreads / 64;
constexpr int kResStep = 256;  // tokens per wave step: 4 rows of 64
constexpr int kResSteps = 8;   // steps per wave at most (4 keys per lane and step in registers)
constexpr int32_t kResCapacity = kResWaves * kResStep * kResSteps;  // 32,768 tokens
static_assert(kResCapacity == kSelResidentCapacity, "host and kernel capacities differ");

struct ResShared {
  uint32_t hist[2048];
  int32_t fstart[kSelFrames];
  int32_t fend[kSelFrames];
  int32_t wlt[kResWaves], weq[kResWaves], wout[kResWaves], weqb[kResWaves];
  int32_t piv_bin, piv_rem;
};

// Classes of the lane's four tokens base + lane + 64 e (e = 0..3) of the wave
// step starting at segment token `base`; cur is the wave-uniform frame cursor.
template <bool LDS>
__device__ __forceinline__ void res_classify(const SeqFrames<LDS>& fr, int32_t& cur, int32_t s0, int32_t base,
                                             int (&cls)[4]) {
  const int lane = threadIdx.x & 63;
  const StepFrames st = step_frames(fr, cur, s0 + base, kResStep);
  const int u = st.n >= 0 ? st.uniform(s0 + base, kResStep) : -1;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int32_t t = s0 + base + 64 * e + lane;
    cls[e] = u >= 0 ? u : (st.n >= 0 ? st.cls(t) : tok_class_search(fr, t));
  }
}

// Bin of the LDS histogram (NB bins, NB a multiple of 64) holding rank k_rem
// (1-based) of the counted keys, and the rank inside it; wave 0 computes it,
// every thread gets it.  The caller synchronised after the counting.
template <int NB>
__device__ __forceinline__ void res_pivot(ResShared& sh, int32_t k_rem, int32_t* bin, int32_t* rem) {
  constexpr int PER = NB / 64;
  const int lane = threadIdx.x & 63;
  if (threadIdx.x < 64) {
    int32_t c = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) c += int32_t(sh.hist[lane * PER + j]);
    const int32_t incl = wave_inscan(c);
    const uint64_t m = __ballot(incl >= k_rem);
    const int L = m ? __ffsll((unsigned long long)m) - 1 : 63;
    if (lane == L) {
      int32_t run = incl - c;
      int b = lane * PER + PER - 1, r = k_rem - run;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int32_t h = int32_t(sh.hist[lane * PER + j]);
        if (run + h >= k_rem) {
          b = lane * PER + j;
          r = k_rem - run;
          break;
        }
        run += h;
      }
      sh.piv_bin = b;
      sh.piv_rem = r;
    }
  }
  __syncthreads();
  *bin = sh.piv_bin;
  *rem = sh.piv_rem;
}

// The selection.  Prod provides
//   Raw;  void load(int32_t base, Raw&)            inputs of tokens base + lane + 64 e;
//   void keys(int32_t base, const int (&cls)[4], int32_t hi, const Raw&, uint32_t (&key)[4])
//        their keys (kSelNever at or past hi and for tokens never selected),
//        writing any per-token output of the pass;
//   void emit(int32_t i, int cls, bool take, int32_t pos)   every token of the range, in order;
//   bool needs_class                                whether keys and emit use the token classes.
// c.k keys are selected; returns T (valid when c.k > 0).
template <class Prod>
__device__ __forceinline__ uint32_t res_select(const Prod& p, ResShared& sh, const SeqFrames<true>& fr,
                                               const SelCtx& c) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  const int32_t R = ((c.n + kResWaves * kResStep - 1) / (kResWaves * kResStep)) * kResStep;
  const int32_t lo = __builtin_amdgcn_readfirstlane(min(wave * R, c.n));
  const int32_t hi = __builtin_amdgcn_readfirstlane(min(lo + R, c.n));
  const int32_t nsteps = __builtin_amdgcn_readfirstlane((hi - lo + kResStep - 1) / kResStep);
  const int32_t cur0 = p.needs_class ? __builtin_amdgcn_readfirstlane(fr.find(c.s0 + lo)) : -1;

  for (int b = threadIdx.x; b < 2048; b += kResThreads) sh.hist[b] = 0u;
  __syncthreads();

  // 1. keys and the histogram of their top 11 bits
  uint32_t key[kResSteps][4];
  {
    typename Prod::Raw raw[2];
    int32_t cur = cur0;
    if (nsteps > 0) p.load(lo, raw[0]);
#pragma unroll
    for (int s = 0; s < kResSteps; ++s) {
#pragma unroll
      for (int e = 0; e < 4; ++e) key[s][e] = kSelNever;
      if (s < nsteps) {
        const int32_t base = lo + s * kResStep;
        if (s + 1 < nsteps) p.load(base + kResStep, raw[(s + 1) & 1]);
        int cls[4] = {kText, kText, kText, kText};
        if (p.needs_class) res_classify(fr, cur, c.s0, base, cls);
        p.keys(base, cls, hi, raw[s & 1], key[s]);
#pragma unroll
        for (int e = 0; e < 4; ++e) sel_hist_add<1>(sh.hist, key[s][e] != kSelNever, key[s][e] >> 21);
      }
    }
  }
  __syncthreads();
  const int32_t k = c.k;
  uint32_t T = 0u;
  int32_t need = 0;
  if (k > 0) {
    // 2. the 11-bit pivot bin, then bits 20..10 and 9..0 of the keys matching the prefix
    int32_t b0, rem0;
    res_pivot<2048>(sh, k, &b0, &rem0);
    for (int b = threadIdx.x; b < 2048; b += kResThreads) sh.hist[b] = 0u;
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kResSteps; ++s) {
      if (s < nsteps) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sel_hist_add<1>(sh.hist, key[s][e] != kSelNever && (key[s][e] >> 21) == uint32_t(b0),
                          (key[s][e] >> 10) & 2047u);
      }
    }
    __syncthreads();
    int32_t b1, rem1;
    res_pivot<2048>(sh, rem0, &b1, &rem1);
    const uint32_t p22 = (uint32_t(b0) << 11) | uint32_t(b1);
    for (int b = threadIdx.x; b < 1024; b += kResThreads) sh.hist[b] = 0u;
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kResSteps; ++s) {
      if (s < nsteps) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sel_hist_add<1>(sh.hist, key[s][e] != kSelNever && (key[s][e] >> 10) == p22, key[s][e] & 1023u);
      }
    }
    __syncthreads();
    int32_t b2, rem2;
    res_pivot<1024>(sh, rem1, &b2, &rem2);
    T = (p22 << 10) | uint32_t(b2);
    need = rem2;
  }

  // 3. counts below and equal to T per wave, their scan, then the ranked walk
  int32_t lt = 0, eqn = 0;
#pragma unroll
  for (int s = 0; s < kResSteps; ++s) {
    if (s < nsteps) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {  // kSelNever is never below T and never equal to it when k > 0
        lt += (k > 0 && key[s][e] < T) ? 1 : 0;
        eqn += (k > 0 && key[s][e] == T) ? 1 : 0;
      }
    }
  }
  lt = wave_sum(lt);
  eqn = wave_sum(eqn);
  if (lane == 0) {
    sh.wlt[wave] = lt;
    sh.weq[wave] = eqn;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t out = 0, eq_before = 0;
    for (int w = 0; w < kResWaves; ++w) {
      sh.wout[w] = out;
      sh.weqb[w] = eq_before;
      out += sh.wlt[w] + min(max(need - eq_before, 0), sh.weq[w]);
      eq_before += sh.weq[w];
    }
  }
  __syncthreads();
  int32_t out = sh.wout[wave], eq_rank = sh.weqb[wave];
  int32_t cur = cur0;
#pragma unroll
  for (int s = 0; s < kResSteps; ++s) {
    if (s < nsteps) {
      const int32_t base = lo + s * kResStep;
      int cls[4] = {kText, kText, kText, kText};
      if (p.needs_class) res_classify(fr, cur, c.s0, base, cls);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool less = k > 0 && key[s][e] < T;
        const bool eq = k > 0 && key[s][e] == T;
        const uint64_t beq = __ballot(eq);
        const bool take = less || (eq && eq_rank + __popcll(beq & below) < need);
        eq_rank += __popcll(beq);
        const uint64_t btk = __ballot(take);
        const int32_t i = base + 64 * e + lane;
        if (i < hi) p.emit(i, cls[e], take, out + __popcll(btk & below));
        out += __popcll(btk);
      }
    }
  }
  return T;
}

}  // namespace stlite
