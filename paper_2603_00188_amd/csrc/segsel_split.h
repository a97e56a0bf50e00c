// Exact k-smallest selection of long segments through splitters drawn from a
// sample.
//
// Same keys, order and result as segsel.h: 32-bit order keys, the k keys first
// in (key ascending, index ascending) order.  Launches:
//   sample    one work-group per segment draws 2048 keys, one from each of
//             2048 equal strata of the segment at a hashed offset, and takes
//             as splitters lo <= hi the sample's exact order statistics five
//             binomial standard deviations (plus 8 ranks) either side of the
//             expected sample rank of the k-th key.  A segment whose k covers
//             every selectable token is marked "all";
//   classify  the whole GPU computes every key once, classifies it against
//             the splitters (below lo, equal to lo, strictly between, equal to
//             hi, above hi, never selected), keeps the four counts of each
//             256-token tile and appends the (key, token) pairs strictly
//             between the splitters to the segment's candidate list (staged
//             per wave in LDS, one global atomic per flush).  A call with a
//             per-token output (the gate) writes it here for every token whose
//             fate the splitters decide; a call with a ranked output list (the
//             top-B) writes a one-byte code per token;
//   resolve   one work-group per segment locates the k-th key T from the tile
//             counts: it is lo or hi (the tied tokens taken are the first ones
//             in index order, up to a cut token) or a candidate (a three-level
//             radix select over the list, held in registers).  It then settles
//             the tokens the splitters left open: the candidates (their output
//             bytes, or their codes), the tied tokens of a tie at lo or hi, and
//             for a ranked list each tile's output offset.  When the splitters
//             miss T or the list overflowed, the work-group selects exactly by
//             streaming the segment itself;
//   emit      (ranked lists only) the whole GPU writes each tile's taken
//             tokens at their ranks.
// The inputs are read once for the keys (twice for a ranked list's codes) and
// no key is stored.  Deterministic: the sample positions are a fixed hash and
// the candidate order (set by atomics) does not change the result.
#pragma once

#include <limits.h>

#include "segsel.h"

namespace stlite {

constexpr int kSpTile = 256;                 // tokens per tile: 4 rows of 64, one wave step
constexpr int kSpThreads = 1024;             // sample and resolve: one work-group per segment
constexpr int kSpWaves = kSpThreads / 64;
constexpr int kSpPerThread = 24;             // candidate entries per resolving thread and batch
constexpr int kSpBatch = kSpPerThread * kSpThreads;  // 24576
constexpr int kSpSampleEach = 2;             // sample keys per sampling thread
constexpr int kSpSampleLog = 11;
constexpr int kSpSample = kSpThreads * kSpSampleEach;  // 2048 sample keys
static_assert(kSpSample == 1 << kSpSampleLog, "the strata are found by a shift");
constexpr int kSpPassThreads = 256;          // classify and emit: 4 waves per work-group
constexpr int kSpPassWaves = kSpPassThreads / 64;
constexpr int kSpStage = 512;                // candidates staged per wave before a flush
constexpr int kSpEmitBatch = 8;              // tiles whose codes an emitting wave loads at once
constexpr int kSpLdsTiles = 4096;            // tiles whose taken counts resolve keeps in LDS (1M tokens)
constexpr uint32_t kSpUniform = 0x100u;      // FrameWin::tile: every token of the tile has one class

// Token codes against the splitters: the number of the four tests key >= lo,
// key > lo, key >= hi, key > hi that hold, plus one for a key never selected
// (above every hi); kCodeTake / kCodeDrop are written by resolve.
enum : uint32_t {
  kCodeLess = 0, kCodeEqLo = 1, kCodeMid = 2, kCodeEqHi = 3, kCodeAbove = 4, kCodeNever = 5, kCodeTake = 6,
  kCodeDrop = 7
};
// Segment modes: kModeNone (k = 0), kModeAll (k covers every selectable token)
// and kModeOpen are set by sample; resolve replaces kModeOpen by how it found T.
enum : int32_t {
  kModeNone = 0, kModeTieLo = 1, kModeMid = 2, kModeTieHi = 3, kModeExact = 4, kModeAll = 5, kModeOpen = 6
};
// Segment state words.
enum : int { kSpLo = 0, kSpHi, kSpK, kSpCount, kSpMode, kSpT, kSpCut, kSpNeed, kSpLe, kSpEqLo, kSpEqHi };
// (kSpLe, kSpEqLo, kSpEqHi: the segment's totals of keys <= lo, == lo and
// == hi, summed by classify.)
// Tile record words: counts of codes 0..3, taken candidates, output offset,
// and (kModeAll) the largest selectable key plus one (0: none).
enum : int { kTileLess = 0, kTileEqLo, kTileMid, kTileEqHi, kTileTaken, kTileOut, kTileMax, kTileWords = 8 };

// Largest value over the wave (DPP within rows, then the row broadcasts).
__device__ __forceinline__ uint32_t sp_wave_max(uint32_t x) {
  x = max(x, uint32_t(__builtin_amdgcn_update_dpp(0, int32_t(x), 0x111, 0xf, 0xf, false)));
  x = max(x, uint32_t(__builtin_amdgcn_update_dpp(0, int32_t(x), 0x112, 0xf, 0xf, false)));
  x = max(x, uint32_t(__builtin_amdgcn_update_dpp(0, int32_t(x), 0x114, 0xf, 0xf, false)));
  x = max(x, uint32_t(__builtin_amdgcn_update_dpp(0, int32_t(x), 0x118, 0xf, 0xf, false)));
  x = max(x, uint32_t(__builtin_amdgcn_update_dpp(0, int32_t(x), 0x142, 0xa, 0xf, false)));
  x = max(x, uint32_t(__builtin_amdgcn_update_dpp(0, int32_t(x), 0x143, 0xc, 0xf, false)));
  return uint32_t(__builtin_amdgcn_readlane(int32_t(x), 63));
}

// A fixed integer hash (the "lowbias32" mix).
__device__ __forceinline__ uint32_t sp_hash(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

__device__ inline int32_t* sp_state(const SelPlan& s, const Layout& lay) { return s.sstate + sel_seg(lay) * kSpWords; }

__device__ inline int32_t* sp_tiles(const SelPlan& s, const Layout& lay, const SelCtx& c) {
  return s.tiles +
         (size_t(blockIdx.z) * sp_tile_stride(lay.total_tokens, lay.n_seqs) + sp_tile_base(c.s0, c.seq)) * kTileWords;
}

__device__ inline uint2* sp_cands(const SelPlan& s, const Layout& lay, const SelCtx& c, int32_t* cap) {
  const int64_t b0 = sp_cand_base(c.s0, c.seq);
  *cap = int32_t(sp_cand_base(int64_t(c.s0) + c.n, c.seq + 1) - b0);
  return s.cands + size_t(blockIdx.z) * sp_cand_stride(lay.total_tokens, lay.n_seqs) + b0;
}

// The segment's codes, one 256-byte block per tile: the code of token
// t * 256 + 64 e + l sits at byte t * 256 + 4 l + e, so a lane reads or writes
// the codes of its four tokens of a tile as one dword.
__device__ inline __amdgpu_buffer_rsrc_t sp_codes(const SelPlan& s, const Layout& lay, const SelCtx& c) {
  const int32_t ntile = (c.n + kSpTile - 1) / kSpTile;
  uint8_t* base = s.codes +
                  (size_t(blockIdx.z) * sp_tile_stride(lay.total_tokens, lay.n_seqs) + sp_tile_base(c.s0, c.seq)) * kSpTile;
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, ntile * kSpTile, kBufferFlags);
}

__device__ __forceinline__ int32_t sp_code_off(int32_t i) { return (i & ~255) | ((i & 63) << 2) | ((i >> 6) & 3); }

// Inclusive scan over the wave with DPP: within rows of 16 lanes, then across
// rows by the row broadcasts of lanes 15 and 31.
__device__ __forceinline__ int32_t sp_wave_inscan(int32_t x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2 and 3
  return x;
}

// Block-wide inclusive scan of one value per thread (kSpThreads threads);
// *total gets the block's sum.  Uses wtot[kSpWaves]; synchronises.
__device__ __forceinline__ int32_t sp_block_inscan(int32_t v, int32_t* wtot, int32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t incl = sp_wave_inscan(v);
  if (lane == 63) wtot[wave] = incl;
  __syncthreads();
  const int32_t t = lane < kSpWaves ? wtot[lane] : 0;
  const int32_t ts = sp_wave_inscan(t);  // lane w: the waves up to w
  const int32_t before = wave > 0 ? __builtin_amdgcn_readlane(ts, wave - 1) : 0;
  *total = __builtin_amdgcn_readlane(ts, kSpWaves - 1);
  __syncthreads();  // wtot is free again
  return incl + before;
}

// The same scan without the closing barrier: the caller synchronises before
// wtot is written again.
__device__ __forceinline__ int32_t sp_block_inscan1(int32_t v, int32_t* wtot, int32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t incl = sp_wave_inscan(v);
  if (lane == 63) wtot[wave] = incl;
  __syncthreads();
  const int32_t t = lane < kSpWaves ? wtot[lane] : 0;
  const int32_t ts = sp_wave_inscan(t);
  const int32_t before = wave > 0 ? __builtin_amdgcn_readlane(ts, wave - 1) : 0;
  *total = __builtin_amdgcn_readlane(ts, kSpWaves - 1);
  return incl + before;
}

// Bins of two 2048-bin LDS histograms holding ranks ra of ha and rb of hb
// (1-based; a rank of 0 is not looked for), and the ranks inside them, to
// out[0..1] and out[2..3], from one scan: thread t takes bins 2t and 2t + 1 of
// both, their sums packed in the halves of one word (every histogram here
// counts fewer than 65536 keys).  The caller synchronised after the
// counting; returns after a barrier.
__device__ __forceinline__ void sp_pivot2(const uint32_t* ha, int32_t ra, const uint32_t* hb, int32_t rb,
                                          int32_t* wtot, int32_t* out) {
  const int32_t t = threadIdx.x;
  const int32_t a0 = int32_t(ha[2 * t]), a1 = int32_t(ha[2 * t + 1]);
  const int32_t b0 = int32_t(hb[2 * t]), b1 = int32_t(hb[2 * t + 1]);
  int32_t total;
  const int32_t incl = sp_block_inscan1((a0 + a1) | ((b0 + b1) << 16), wtot, &total);
  const int32_t ia = incl & 0xffff, ib = incl >> 16;
  const int32_t fa = ia - a0 - a1, fb = ib - b0 - b1;
  if (ra > 0 && ia >= ra && fa < ra) {
    out[0] = fa + a0 >= ra ? 2 * t : 2 * t + 1;
    out[1] = fa + a0 >= ra ? ra - fa : ra - fa - a0;
  }
  if (rb > 0 && ib >= rb && fb < rb) {
    out[2] = fb + b0 >= rb ? 2 * t : 2 * t + 1;
    out[3] = fb + b0 >= rb ? rb - fb : rb - fb - b0;
  }
  __syncthreads();
}

// One histogram's pivot as in sp_pivot2, plus the count of the bin found
// (out[2]).
__device__ __forceinline__ void sp_pivot1(const uint32_t* h, int32_t r, int32_t* wtot, int32_t* out) {
  const int32_t t = threadIdx.x;
  const int32_t h0 = int32_t(h[2 * t]), h1 = int32_t(h[2 * t + 1]);
  int32_t total;
  const int32_t incl = sp_block_inscan1(h0 + h1, wtot, &total);
  const int32_t f = incl - h0 - h1;
  if (incl >= r && f < r) {
    const bool first = f + h0 >= r;
    out[0] = first ? 2 * t : 2 * t + 1;
    out[1] = first ? r - f : r - f - h0;
    out[2] = first ? h0 : h1;
  }
  __syncthreads();
}

// sp_pivot1 over a histogram of `bins` bins (a power of two, at most 8
// kSpThreads): thread t sums bins [t w, t w + w), w = bins / kSpThreads or 1,
// and the thread holding rank r walks its own.
__device__ __forceinline__ void sp_pivot_wide(const uint32_t* h, int32_t bins, int32_t r, int32_t* wtot,
                                              int32_t* out) {
  const int32_t t = threadIdx.x;
  const int32_t w = bins > kSpThreads ? bins / kSpThreads : 1;
  const int32_t b0 = t * w;
  int32_t sum = 0;
  if (w == 8) {
    const uint4 x = *reinterpret_cast<const uint4*>(h + b0), y = *reinterpret_cast<const uint4*>(h + b0 + 4);
    sum = int32_t(x.x + x.y + x.z + x.w + y.x + y.y + y.z + y.w);
  } else if (b0 < bins) {
    for (int32_t j = 0; j < w; ++j) sum += int32_t(h[b0 + j]);
  }
  int32_t total;
  const int32_t incl = sp_block_inscan1(sum, wtot, &total);
  int32_t f = incl - sum;
  if (b0 < bins && incl >= r && f < r) {
    int32_t j = 0;
    for (; j + 1 < w; ++j) {
      const int32_t x = int32_t(h[b0 + j]);
      if (f + x >= r) break;
      f += x;
    }
    out[0] = b0 + j;
    out[1] = r - f;
    out[2] = int32_t(h[b0 + j]);
  }
  __syncthreads();
}

// Bin of a 2048-bin LDS histogram holding rank r (1-based) of its counts, and
// the rank inside it, to out[0..1]: thread t scans bins 2t and 2t + 1 (a
// kSpThreads-thread block).  The caller synchronised after the counting;
// returns after a barrier.
__device__ __forceinline__ void sp_pivot(const uint32_t* hist, int32_t r, int32_t* wtot, int32_t* out) {
  const int32_t t = threadIdx.x;
  const int32_t h0 = int32_t(hist[2 * t]), h1 = int32_t(hist[2 * t + 1]);
  int32_t total;
  const int32_t incl = sp_block_inscan(h0 + h1, wtot, &total);
  const int32_t before = incl - h0 - h1;
  if (incl >= r && before < r) {
    if (before + h0 >= r) {
      out[0] = 2 * t;
      out[1] = r - before;
    } else {
      out[0] = 2 * t + 1;
      out[1] = r - before - h0;
    }
  }
  __syncthreads();
}

// Device-scope load that bypasses the vector L1 (values written by atomics).
__device__ __forceinline__ int32_t sp_load_agent(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Token classes of whole tiles from a window of 64 frames held in registers
// (lane l: frame f0 + l of the sequence, absolute [s, e)), moved forward as a
// wave's tiles advance; frames are disjoint and in token order.  A tile is
// classified by one ballot of the frames overlapping it; a tile that overlaps
// more frames than the window holds falls back to a search per token.
struct FrameWin {
  const int32_t* meta;  // frame_meta rows of the sequence's frames
  int32_t nf;
  int32_t f0;
  int32_t s, e;

  __device__ void load(int32_t f) {
    f0 = f;
    const int32_t g = f + int32_t(threadIdx.x & 63);
    s = e = INT_MAX;
    if (g < nf) {
      const int32_t* m = meta + 3 * g;
      s = m[0];
      e = m[0] + m[1] * m[2];
    }
  }

  // A window whose frames before f0 end at or before token tok.
  __device__ void init(const Layout& lay, int32_t seq, int32_t tok) {
    const int32_t g0 = lay.cu_frames[seq];
    meta = lay.frame_meta + 3 * g0;
    nf = lay.cu_frames[seq + 1] - g0;
    int32_t f = 0;
    if (nf > 64) {  // the last frame starting at or before tok
      int32_t lo = 0, hi = nf - 1;
      f = -1;
      while (lo <= hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (meta[3 * mid] <= tok) {
          f = mid;
          lo = mid + 1;
        } else {
          hi = mid - 1;
        }
      }
      f = max(f, 0);
    }
    load(f);
  }

  // Classes of tokens b + 64 q + lane (q = 0..3) of the tile starting at
  // absolute token b, two bits per token at bit 2 q: bit 0 the token lies in
  // a frame, bit 1 in the sequence's last (current) frame; kSpUniform is set
  // when every token of the tile has the same class.  Tiles come in
  // increasing order.  Wave-uniform.
  __device__ uint32_t tile(int32_t b) {
    const int lane = threadIdx.x & 63;
    const int32_t last = b + kSpTile;
    bool search = false;
    for (;;) {  // slide until no frame past the window can overlap the tile
      const int32_t s63 = __builtin_amdgcn_readlane(s, 63);
      if (s63 >= last) break;  // INT_MAX: past the sequence's frames
      const int32_t drop = __popcll(__ballot(e <= b));
      if (drop == 0) {
        search = true;  // more than 64 frames overlap the tile
        break;
      }
      load(f0 + drop);
    }
    uint32_t bits = 0u;
    if (search) {
      for (int q = 0; q < 4; ++q) {
        const int32_t tok = b + 64 * q + lane;
        int32_t lo = 0, hi = nf - 1, f = -1;
        while (lo <= hi) {
          const int32_t mid = (lo + hi) >> 1;
          if (meta[3 * mid] <= tok) {
            f = mid;
            lo = mid + 1;
          } else {
            hi = mid - 1;
          }
        }
        if (f >= 0 && tok < meta[3 * f] + meta[3 * f + 1] * meta[3 * f + 2]) bits |= (f == nf - 1 ? 3u : 1u) << (2 * q);
      }
      return bits;
    }
    uint64_t m = __ballot(s < last && e > b);
    if (m == 0) return kSpUniform;  // text only
    if ((m & (m - 1)) == 0) {       // one frame: uniform when it covers the tile
      const int j = __ffsll((unsigned long long)m) - 1;
      if (__builtin_amdgcn_readlane(s, j) <= b && __builtin_amdgcn_readlane(e, j) >= last)
        return kSpUniform | (f0 + j == nf - 1 ? 0xffu : 0x55u);
    }
    while (m) {  // few frames overlap one tile
      const int j = __ffsll((unsigned long long)m) - 1;
      m &= m - 1;
      const int32_t sf = __builtin_amdgcn_readlane(s, j), ef = __builtin_amdgcn_readlane(e, j);
      const uint32_t c = f0 + j == nf - 1 ? 3u : 1u;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int32_t tok = b + 64 * q + lane;
        bits |= (tok >= sf && tok < ef) ? c << (2 * q) : 0u;
      }
    }
    return bits;
  }
};

// Token class (kText, kHist, kCurrent) of token q from FrameWin::tile bits.
// (kSpUniform, bit 8 of those bits, is above every token's pair.)
__device__ __forceinline__ int sp_cls(uint32_t bits, int q) {
  const uint32_t b = (bits >> (2 * q)) & 3u;
  return int((b & 1u) + (b >> 1));
}

// The keys of the lane's four tokens of tile t (tokens of a wave's tiles in
// increasing order: the frame window moves forward).
template <class Prod>
__device__ __forceinline__ void sp_tile_keys(const Prod& p, FrameWin& win, const SelCtx& c, int32_t t,
                                             uint32_t (&key)[4]) {
  typename Prod::Raw raw;
  p.load(t * kSpTile, raw);
  const uint32_t cb = p.needs_class ? win.tile(c.s0 + t * kSpTile) : 0u;
  int cls[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) cls[q] = sp_cls(cb, q);
  p.keys(t * kSpTile, cls, c.n, raw, key);
}

// ---------------------------------------------------------------------------
// sample: splitters of one segment (grid (1, seqs, units), kSpThreads threads)
// ---------------------------------------------------------------------------

struct SpSampleShared {
  uint32_t hist[2][2][2048];  // two sets (alternate levels) of the lo and hi histograms
  int32_t fstart[kSelFrames];
  int32_t fend[kSelFrames];
  int32_t wtot[kSpWaves];
  int32_t piv[4];
};

// The sample positions of one segment and the first step of their loads,
// issued before anything else of the sample kernel: the n tokens fall in
// S = min(2048, n) strata [floor(j n / S), floor((j + 1) n / S)), and stratum j
// (thread j mod kSpThreads, slot j / kSpThreads) gives one hashed position.
// Prod provides Raw1, void load1(int32_t i, Raw1&), void load1_rest(int32_t
// i, int cls, Raw1&) and uint32_t key1(const Raw1&, int cls): the inputs of
// segment token i, in two steps (the second may skip what the first and the
// class make unneeded), and its key; needs_class.
template <class Prod>
struct SpGather {
  uint32_t valid;
  int32_t pos[kSpSampleEach];
  typename Prod::Raw1 raw[kSpSampleEach];
};

template <class Prod>
__device__ __forceinline__ void sp_gather(const Prod& p, const Layout& lay, const SelCtx& c, SpGather<Prod>& g) {
  const int32_t n = c.n, S = min(kSpSample, n);
  const uint32_t salt = sp_hash(uint32_t(sel_seg(lay)) * 0x9e3779b9u + 0x51ed27u);
  g.valid = 0u;
#pragma unroll
  for (int e = 0; e < kSpSampleEach; ++e) {
    const int32_t j = int32_t(threadIdx.x) + kSpThreads * e;
    g.pos[e] = 0;
    if (j < S) {
      const int32_t a = S == n ? j : int32_t((int64_t(j) * n) >> kSpSampleLog);
      const int32_t b = S == n ? j + 1 : int32_t((int64_t(j + 1) * n) >> kSpSampleLog);
      g.pos[e] = a + int32_t(__umulhi(sp_hash(uint32_t(j) ^ salt), uint32_t(b - a)));
      g.valid |= 1u << e;
    }
    p.load1(g.pos[e], g.raw[e]);  // position 0 of an empty segment reads 0 (buffer bounds)
  }
}

// c.k keys are to be selected among n_sel selectable tokens, from the sample
// sp_gather started.  Writes lo, hi, k, the mode and a zero candidate count.
template <class Prod, bool LDS>
__device__ void split_sample(const Prod& p, SpSampleShared& sh, const SeqFrames<LDS>& fr, const SelPlan& s,
                             const Layout& lay, const SelCtx& c, int32_t n_sel, SpGather<Prod>& g) {
  int32_t* st = sp_state(s, lay);
  const int32_t n = c.n, k = c.k;
  if (threadIdx.x == 0) {
    st[kSpLe] = 0;
    st[kSpEqLo] = 0;
    st[kSpEqHi] = 0;
  }
  if (Prod::kDirect) {  // classify writes the records of tiles with ties (or of every tile in kModeAll)
    int32_t* tiles = sp_tiles(s, lay, c);
    const int32_t ntile = (n + kSpTile - 1) / kSpTile;
    for (int32_t i = threadIdx.x; i < ntile * (kTileWords / 4); i += kSpThreads)
      reinterpret_cast<int4*>(tiles)[i] = make_int4(0, 0, 0, 0);
  }
  if (n <= 0 || k <= 0 || k >= n_sel) {
    if (threadIdx.x == 0) {
      st[kSpLo] = 0;
      st[kSpHi] = 0;
      st[kSpK] = max(k, 0);
      st[kSpCount] = 0;
      st[kSpMode] = (n <= 0 || k <= 0) ? kModeNone : kModeAll;
    }
    return;
  }
  const int32_t S = min(kSpSample, n);
  const uint32_t valid = g.valid;
  const int32_t (&pos)[kSpSampleEach] = g.pos;
  typename Prod::Raw1 (&raw)[kSpSampleEach] = g.raw;
  uint32_t key[kSpSampleEach];
  int cls[kSpSampleEach];
#pragma unroll
  for (int e = 0; e < kSpSampleEach; ++e) cls[e] = kText;
  if (p.needs_class && fr.nf > 0) {
    // frame of each sample: a branchless search, the lookups of a step together
    int32_t f[kSpSampleEach];
#pragma unroll
    for (int e = 0; e < kSpSampleEach; ++e) f[e] = -1;
    int32_t step = 1;
    while (step * 2 <= fr.nf) step *= 2;
    for (; step > 0; step >>= 1) {
#pragma unroll
      for (int e = 0; e < kSpSampleEach; ++e) {
        const int32_t g = f[e] + step;
        if (g < fr.nf && fr.start(g) <= c.s0 + pos[e]) f[e] = g;
      }
    }
#pragma unroll
    for (int e = 0; e < kSpSampleEach; ++e)
      if (f[e] >= 0 && c.s0 + pos[e] < fr.end(f[e])) cls[e] = f[e] == fr.nf - 1 ? kCurrent : kHist;
  }
#pragma unroll
  for (int e = 0; e < kSpSampleEach; ++e) p.load1_rest(pos[e], cls[e], raw[e]);
#pragma unroll
  for (int e = 0; e < kSpSampleEach; ++e) key[e] = ((valid >> e) & 1u) ? p.key1(raw[e], cls[e]) : kSelNever;
  // the sample keys of ranks qlo and qhi (1-based), exactly: three radix levels
  const double pr = double(k) / double(n);
  const int32_t delta = int32_t(ceil(5.0 * sqrt(double(S) * pr * (1.0 - pr)))) + 8;
  const int32_t rt = int32_t(double(k) * double(S) / double(n));
  int32_t rlo = rt - delta, rhi = rt + delta;
  const bool has_lo = rlo >= 1, has_hi = rhi <= S;
  uint32_t plo = 0u, phi = 0u;  // the two keys' prefixes so far
  for (int b = threadIdx.x; b < 2 * 2048; b += kSpThreads) (&sh.hist[0][0][0])[b] = 0u;
  __syncthreads();
#pragma unroll 1
  for (int level = 0; level < 3; ++level) {
    const int shift = level == 0 ? 21 : level == 1 ? 10 : 0;
    const uint32_t mask = level == 2 ? 1023u : 2047u;
    const int pshift = level == 1 ? 21 : 10;
    uint32_t* hlo = sh.hist[level & 1][0];
    uint32_t* hhi = sh.hist[level & 1][1];
    // level 0 counts every key once (both ranks pivot on it); levels 1 and 2
    // the keys matching each rank's prefix
#pragma unroll
    for (int e = 0; e < kSpSampleEach; ++e) {
      if (!((valid >> e) & 1u)) continue;
      const uint32_t d = (key[e] >> shift) & mask;
      if (level == 0 || (has_lo && (key[e] >> pshift) == (plo >> pshift))) atomicAdd(&hlo[d], 1u);
      if (level > 0 && has_hi && (key[e] >> pshift) == (phi >> pshift)) atomicAdd(&hhi[d], 1u);
    }
    // the other set, read by the previous level's pivots, is cleared for the next level
    for (int b = threadIdx.x; b < 2 * 2048; b += kSpThreads) (&sh.hist[(level + 1) & 1][0][0])[b] = 0u;
    __syncthreads();
    sp_pivot2(hlo, has_lo ? rlo : 0, level == 0 ? hlo : hhi, has_hi ? rhi : 0, sh.wtot, sh.piv);
    if (has_lo) {
      plo |= uint32_t(sh.piv[0]) << shift;
      rlo = sh.piv[1];
    }
    if (has_hi) {
      phi |= uint32_t(sh.piv[2]) << shift;
      rhi = sh.piv[3];
    }
  }
  if (threadIdx.x == 0) {
    // The two splitters are kept distinct: a key equal to both would take the
    // code of a key strictly between them while counting as a tie at both
    // (a tie group covering the whole sample band, e.g. the gated-out S = 0).
    uint32_t lo = has_lo ? min(plo, kSelKeyMax) : 0u;
    uint32_t hi = has_hi ? min(phi, kSelKeyMax) : kSelKeyMax;
    if (lo == hi) {
      if (hi < kSelKeyMax) hi = lo + 1u;
      else lo = hi - 1u;
    }
    st[kSpLo] = int32_t(lo);
    st[kSpHi] = int32_t(hi);
    st[kSpK] = k;
    st[kSpCount] = 0;
    st[kSpMode] = kModeOpen;
  }
}

// ---------------------------------------------------------------------------
// classify: codes or direct outputs, tile counts and candidates (grid (parts,
// seqs, units), kSpPassThreads threads)
// ---------------------------------------------------------------------------

struct SpPassShared {
  uint2 stage[kSpPassWaves][kSpStage];
  uint32_t xpose[kSpPassWaves][64];  // a tile's output bytes, from rows to runs of four tokens
};

// Tiles of one work-group of the classify and emit passes: [t0, t1) of the
// segment's ceil(n / 256) tiles; wave w takes t0 + w, t0 + w + 4, ...
__device__ inline void sp_part_tiles(int32_t n, int32_t parts, int32_t part, int32_t* t0, int32_t* t1) {
  const int32_t ntile = (n + kSpTile - 1) / kSpTile;
  const int32_t per = (ntile + parts - 1) / parts;
  *t0 = min(part * per, ntile);
  *t1 = min(*t0 + per, ntile);
}

// Prod as in segsel_resident.h (Raw, load, keys, needs_class), plus kGroup
// (tiles whose inputs a wave loads at once) and kDirect: the call's output is
// one byte per token (Prod::put_byte / put_word, aligned: whether four tokens
// of a tile's run form a 4-byte aligned word), written here from each code:
// 1 for a token never selected, below lo or equal to lo (the taken side when T
// lies above lo), 0 otherwise; resolve settles the rest.  Without kDirect a
// one-byte code per token goes to the codes array.  A wave's tiles go in
// groups of kGroup, the next group's loads in flight while one is classified.
template <class Prod>
__device__ void split_classify(const Prod& p, SpPassShared& sh, const SelPlan& s, const Layout& lay,
                               const SelCtx& c) {
  constexpr int G = Prod::kGroup;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int32_t* st = sp_state(s, lay);
  const uint32_t lo = uint32_t(st[kSpLo]), hi = uint32_t(st[kSpHi]);
  const int32_t mode = st[kSpMode];
  int32_t t0, t1;
  sp_part_tiles(c.n, s.split_parts, c.part, &t0, &t1);
  const int32_t tw = t0 + wave;  // this wave's tiles: tw + 4 j, j < nt
  const int32_t nt = tw < t1 ? (t1 - tw + kSpPassWaves - 1) / kSpPassWaves : 0;
  if (nt == 0) return;
  int32_t* tiles = sp_tiles(s, lay, c);
  int32_t cap;
  uint2* cands = sp_cands(s, lay, c, &cap);
  const __amdgpu_buffer_rsrc_t codes = sp_codes(s, lay, c);
  uint2* stage = sh.stage[wave];
  uint8_t* xb = reinterpret_cast<uint8_t*>(sh.xpose[wave]);
  int32_t staged = 0;
  auto flush = [&]() {
    int32_t b = 0;
    if (lane == 0) b = atomicAdd(&st[kSpCount], staged);
    b = __builtin_amdgcn_readfirstlane(b);
    for (int32_t i = lane; i < staged; i += 64)
      if (b + i < cap) cands[b + i] = stage[i];
    staged = 0;
  };
  // the output bytes of one tile (byte e: token base + 64 e + lane)
  auto put = [&](int32_t base, uint32_t bytes) {
    if (p.aligned && base + kSpTile <= c.n) {  // a word of four consecutive tokens per lane
#pragma unroll
      for (int e = 0; e < 4; ++e) xb[64 * e + lane] = uint8_t(bytes >> (8 * e));
      p.put_word(base + 4 * lane, sh.xpose[wave][lane]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (base + 64 * e + lane < c.n) p.put_byte(base + 64 * e + lane, uint8_t(bytes >> (8 * e)));
    }
  };
  FrameWin win;
  if (p.needs_class) win.init(lay, c.seq, c.s0 + tw * kSpTile);
  // Class facts of a group's tiles, wave-uniform where a tile has one class:
  // uni bit i: tile i has one class and no token past the segment; ucls bits
  // 2i..2i+1: that class; cb: per-lane class bits (eight per tile) of the
  // others.  Called for the groups in order (the frame window moves forward).
  struct GroupCls {
    uint32_t cb, uni, ucls;
  };
  auto classes = [&](int32_t j0) {
    GroupCls g{0u, 0u, 0u};
#pragma unroll 1
    for (int i = 0; i < G; ++i) {
      if (j0 + i >= nt) break;
      const int32_t base = (tw + kSpPassWaves * (j0 + i)) * kSpTile;
      const uint32_t x = p.needs_class ? win.tile(c.s0 + base) : kSpUniform;  // no class needed: "text"
      if ((x & kSpUniform) && base + kSpTile <= c.n) {
        g.uni |= 1u << i;
        g.ucls |= uint32_t(__builtin_amdgcn_readfirstlane(sp_cls(x, 0))) << (2 * i);
      }
      g.cb |= (x & 0xffu) << (8 * i);
    }
    g.uni = __builtin_amdgcn_readfirstlane(g.uni);
    g.ucls = __builtin_amdgcn_readfirstlane(g.ucls);
    return g;
  };
  auto fetch = [&](typename Prod::Raw (&raw)[G], int32_t j0, const GroupCls& g) {
#pragma unroll
    for (int i = 0; i < G; ++i)  // a uniform tile with nothing selectable is not read
      if (j0 + i < nt && !(((g.uni >> i) & 1u) && !p.selectable(int((g.ucls >> (2 * i)) & 3u))))
        p.load((tw + kSpPassWaves * (j0 + i)) * kSpTile, raw[i]);
  };
  // the segment's totals (keys <= lo: for a direct output a per-lane count in
  // the fast path and a wave count elsewhere; ties at lo and at hi)
  uint32_t le_lane = 0u;
  int32_t le_w = 0, eqlo_w = 0, eqhi_w = 0;
  // cnt: keys <= lo, == lo, strictly between, == hi.  A ranked list records
  // every tile; a direct output the tiles with ties (its totals go to the
  // state words) and, in kModeAll, the tiles' largest keys.
  auto finish_tile = [&](int32_t t, int32_t base, uint32_t packed, const int32_t (&cnt)[4], uint32_t kmax) {
    if (Prod::kDirect) put(base, packed);
    else __builtin_amdgcn_raw_buffer_store_b32(packed, codes, base + 4 * lane, 0, 0);
    le_w += cnt[0];
    eqlo_w += cnt[1];
    eqhi_w += cnt[3];
    if (!Prod::kDirect || cnt[1] + cnt[3] > 0 || mode == kModeAll) {
      if (lane == 0) {
        int4* rec = reinterpret_cast<int4*>(tiles + size_t(t) * kTileWords);
        rec[0] = make_int4(Prod::kDirect ? 0 : cnt[0] - cnt[1], cnt[1], cnt[2], cnt[3]);
        rec[1] = make_int4(0, 0, int32_t(kmax), 0);
      }
    }
  };
  // counts and candidates of one row from its tests: cnt[0] gathers the keys
  // at or below lo (the tile's count below lo is cnt[0] - cnt[1] once the
  // tile is done); ties at lo or hi are rare, so their masks are tested first
  auto tally = [&](int e, int32_t base, uint32_t key, bool ge_lo, bool gt_lo, bool ge_hi, bool gt_hi,
                   int32_t (&cnt)[4]) {
    const uint64_t mge_lo = __ballot(ge_lo), mgt_lo = __ballot(gt_lo), mge_hi = __ballot(ge_hi),
                   mgt_hi = __ballot(gt_hi);
    cnt[0] += __popcll(~mgt_lo);
    const uint64_t eq_lo = mge_lo & ~mgt_lo, eq_hi = mge_hi & ~mgt_hi, mid = mgt_lo & ~mge_hi;
    if (eq_lo) cnt[1] += __popcll(eq_lo);
    if (eq_hi) cnt[3] += __popcll(eq_hi);
    if (mid) {
      const int32_t nm = __popcll(mid);
      cnt[2] += nm;
      if (gt_lo && !ge_hi) stage[staged + __popcll(mid & below)] = make_uint2(key, uint32_t(base + 64 * e + lane));
      staged += nm;
    }
  };
  auto process = [&](const typename Prod::Raw (&raw)[G], int32_t j0, const GroupCls& g) {
#pragma unroll
    for (int i = 0; i < G; ++i) {
      if (j0 + i >= nt) break;
      if (staged > kSpStage - kSpTile) flush();
      const int32_t t = tw + kSpPassWaves * (j0 + i);
      const int32_t base = t * kSpTile;
      int32_t cnt[4] = {0, 0, 0, 0};
      uint32_t packed = 0u, kmax = 0u;
      const int ucls = int((g.ucls >> (2 * i)) & 3u);
      if (mode == kModeOpen && ((g.uni >> i) & 1u)) {  // the common case: one class, inside the segment
        if (!p.selectable(ucls)) {                     // nothing selectable: every token "never"
          finish_tile(t, base, Prod::kDirect ? 0x01010101u : kCodeNever * 0x01010101u, cnt, 0u);
          continue;
        }
        uint32_t key[4];
        p.keys_uniform(base, ucls, raw[i], key);
        // every key is selectable here: each test's compare feeds its ballot
        // and the lane's code directly; ties are rare, so their masks are only
        // counted when some row has one
        const int32_t staged0 = staged;
        int32_t gt = 0;  // keys above lo (ranked lists)
        uint64_t eql[4], eqh[4], eq_any = 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t k = key[e];
          const uint64_t mgt_lo = __ballot(k > lo), mlt_hi = __ballot(k < hi);
          eql[e] = __ballot(k == lo);
          eqh[e] = __ballot(k == hi);
          eq_any |= eql[e] | eqh[e];
          uint32_t code;
          if (Prod::kDirect) {
            code = k > lo ? 0u : 1u;
            le_lane += code;
          } else {
            code = (k >= lo ? 1u : 0u) + (k > lo ? 1u : 0u) + (k >= hi ? 1u : 0u) + (k > hi ? 1u : 0u);
            gt += __popcll(mgt_lo);
          }
          packed |= code << (8 * e);
          const uint64_t mid = mgt_lo & mlt_hi;
          const uint32_t rank =
              __builtin_amdgcn_mbcnt_hi(uint32_t(mid >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(mid), 0u));
          if (k > lo && k < hi) stage[staged + int32_t(rank)] = make_uint2(k, uint32_t(base + 64 * e + lane));
          staged += __popcll(mid);
        }
        if (eq_any) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            cnt[1] += __popcll(eql[e]);
            cnt[3] += __popcll(eqh[e]);
          }
        }
        cnt[0] = Prod::kDirect ? 0 : kSpTile - gt;  // direct: these keys are counted in le_lane
        cnt[2] = staged - staged0;
        finish_tile(t, base, packed, cnt, 0u);
        continue;
      }
      uint32_t key[4];
      int cls[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) cls[q] = sp_cls(g.cb >> (8 * i), q);
      p.keys(base, cls, c.n, raw[i], key);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (mode == kModeAll && key[e] != kSelNever) kmax = max(kmax, key[e] + 1u);
        const bool ge_lo = key[e] >= lo, gt_lo = key[e] > lo, ge_hi = key[e] >= hi, gt_hi = key[e] > hi;
        const bool never = key[e] == kSelNever;
        uint32_t code = uint32_t(ge_lo) + uint32_t(gt_lo) + uint32_t(ge_hi) + uint32_t(gt_hi) + uint32_t(never);
        if (Prod::kDirect) code = (never || (mode == kModeAll && base + 64 * e + lane < c.n) ||
                                   (mode == kModeOpen && !gt_lo)) ? 1u : 0u;
        else if (mode == kModeAll) code = never ? kCodeNever : kCodeTake;
        packed |= code << (8 * e);
        if (mode == kModeOpen) tally(e, base, key[e], ge_lo, gt_lo, ge_hi, gt_hi, cnt);
      }
      if (mode == kModeAll) kmax = sp_wave_max(kmax);
      finish_tile(t, base, packed, cnt, kmax);
    }
  };
  typename Prod::Raw ra[G], rb[G];
  GroupCls ga = classes(0), gb{0u, 0u, 0u};
  fetch(ra, 0, ga);
  for (int32_t j = 0; j < nt; j += 2 * G) {
    if (j + G < nt) {
      gb = classes(j + G);
      fetch(rb, j + G, gb);
    }
    process(ra, j, ga);
    if (j + G >= nt) break;
    if (j + 2 * G < nt) {
      ga = classes(j + 2 * G);
      fetch(ra, j + 2 * G, ga);
    }
    process(rb, j + G, gb);
  }
  if (staged) flush();
  {  // the wave's totals
    const int32_t le = __builtin_amdgcn_readlane(sp_wave_inscan(int32_t(le_lane)), 63) + le_w;
    if (lane == 0) {
      if (le) atomicAdd(&st[kSpLe], le);
      if (eqlo_w) atomicAdd(&st[kSpEqLo], eqlo_w);
      if (eqhi_w) atomicAdd(&st[kSpEqHi], eqhi_w);
    }
  }
}

// ---------------------------------------------------------------------------
// resolve: T, the open tokens and the tile offsets of one segment (grid (1,
// seqs, units), kSpThreads threads)
// ---------------------------------------------------------------------------

constexpr int kSpCandBits = 13;  // radix bits per level of the candidate selection
constexpr int kSpCandBins = 1 << kSpCandBits;
constexpr int kSpTieList = 256;  // tied candidates ordered by a direct rank count

struct SpResolveShared {
  uint32_t hist[2048];
  uint32_t hist2[2][kSpCandBins];  // alternate levels of the candidate selection
  int32_t tcount[kSpLdsTiles];  // taken candidates per tile (segments of at most kSpLdsTiles tiles)
  int32_t wtot[kSpWaves];
  int32_t weq[kSpWaves];
  int32_t piv[3];
  int32_t sum[4];
  int32_t found[2];
  int32_t cut;
};

// Exact select of rank r (1-based) among the keys kf(v) of the candidate
// entries held in v (kSpPerThread per thread, batch i0 of the list), reloaded
// per batch by reload(i0) when the list has more than one batch.  Every
// counted key lies in [lo_b, hi_b]: they share the bits above the highest bit
// where lo_b and hi_b differ, and radix levels of up to kSpCandBits bits cover
// the bits below it (so the first level already spreads the keys over its
// bins, and two levels cover 26 varying bits).  kSelNever is not counted.
// Returns T; *need gets its rank among the keys equal to T, *eq how many there
// are.
template <class KeyOf, class Reload>
__device__ uint32_t sp_cand_select(const KeyOf& kf, const Reload& reload, const uint2 (&v)[kSpPerThread],
                                   int32_t count, bool one, int32_t r, uint32_t lo_b, uint32_t hi_b,
                                   SpResolveShared& sh, int32_t* need, int32_t* eq) {
  const uint32_t diff = lo_b ^ hi_b;
  int top = diff ? 32 - __clz(int32_t(diff)) : 0;  // bits [0, top) vary
  uint32_t prefix = top >= 32 ? 0u : lo_b & ~((1u << top) - 1u);
  int32_t rem = r;
  *eq = count;
  int32_t bins = top > 0 ? 1 << min(top, kSpCandBits) : 0;
  for (int b = threadIdx.x; b < bins; b += kSpThreads) sh.hist2[0][b] = 0u;
  __syncthreads();
  int cur = 0;
#pragma unroll 1
  while (top > 0) {
    const int shift = max(top - kSpCandBits, 0);
    const uint32_t mask = (1u << (top - shift)) - 1u;
    uint32_t* h = sh.hist2[cur];
    for (int32_t i0 = 0; i0 < count; i0 += kSpBatch) {
      if (!one) reload(i0);
#pragma unroll
      for (int e = 0; e < kSpPerThread; ++e) {
        const uint32_t key = kf(v[e]);
        if (key != kSelNever && (top >= 32 || (key >> top) == (prefix >> top))) atomicAdd(&h[(key >> shift) & mask], 1u);
      }
    }
    // the other set, read by the previous level's pivot, is cleared for the next level
    const int32_t next = shift > 0 ? 1 << min(shift, kSpCandBits) : 0;
    for (int b = threadIdx.x; b < next; b += kSpThreads) sh.hist2[cur ^ 1][b] = 0u;
    __syncthreads();
    sp_pivot_wide(h, int32_t(mask) + 1, rem, sh.wtot, sh.piv);
    prefix |= uint32_t(sh.piv[0]) << shift;
    rem = sh.piv[1];
    if (shift == 0) *eq = sh.piv[2];
    top = shift;
    cur ^= 1;
  }
  __syncthreads();  // every thread has read the last pivot before sh.piv is reused
  *need = rem;
  return prefix;
}

// Index of the need-th (1-based) candidate, in index order, among the eq
// candidates whose key is T (eq <= kSpTieMax; the indices lie in [0, n)).
// They are gathered in LDS; up to kSpTieList of them rank themselves by a
// direct count, more are selected by radix levels over the gathered indices.
constexpr int kSpTieMax = 2 * kSpCandBins;

template <class Reload>
__device__ int32_t sp_tie_cut(const Reload& reload, const uint2 (&v)[kSpPerThread], int32_t count, bool one,
                              uint32_t T, int32_t need, int32_t eq, int32_t n, SpResolveShared& sh) {
  uint32_t* list = sh.hist2[0];  // both sets: kSpTieMax entries
  const int lane = threadIdx.x & 63;
  if (threadIdx.x == 0) sh.found[0] = 0;
  __syncthreads();
  for (int32_t i0 = 0; i0 < count; i0 += kSpBatch) {
    if (!one) reload(i0);
#pragma unroll
    for (int e = 0; e < kSpPerThread; ++e) {
      const uint64_t m = __ballot(v[e].x == T);
      if (m) {  // the wave's tied entries appended at once
        int32_t b = 0;
        if (lane == 0) b = atomicAdd(&sh.found[0], __popcll(m));
        b = __builtin_amdgcn_readfirstlane(b);
        const uint32_t rank =
            __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
        if (v[e].x == T) list[b + int32_t(rank)] = v[e].y;
      }
    }
  }
  __syncthreads();
  const int32_t m = sh.found[0];  // == eq
  if (m <= kSpTieList) {
    if (int32_t(threadIdx.x) < m) {
      const uint32_t mine = list[threadIdx.x];
      int32_t rank = 1;
      for (int32_t j = 0; j < m; ++j) rank += list[j] < mine ? 1 : 0;
      if (rank == need) sh.cut = int32_t(mine);
    }
    __syncthreads();
    return sh.cut;
  }
  int top = n > 1 ? 32 - __clz(n - 1) : 1;  // index bits [0, top) vary
  uint32_t prefix = 0u;
  int32_t rem = need;
#pragma unroll 1
  while (top > 0) {
    const int shift = max(top - 11, 0);
    const uint32_t mask = (1u << (top - shift)) - 1u;
    for (int b = threadIdx.x; b < 2048; b += kSpThreads) sh.hist[b] = 0u;
    __syncthreads();
    for (int32_t j = threadIdx.x; j < m; j += kSpThreads) {
      const uint32_t x = list[j];
      if ((x >> top) == (prefix >> top)) atomicAdd(&sh.hist[(x >> shift) & mask], 1u);
    }
    __syncthreads();
    sp_pivot(sh.hist, rem, sh.wtot, sh.piv);
    prefix |= uint32_t(sh.piv[0]) << shift;
    rem = sh.piv[1];
    top = shift;
  }
  return int32_t(prefix);
}

// Exact selection by streaming the segment's own inputs (the splitters missed
// T or the candidate list overflowed): T, then every output rewritten (a
// direct output's bytes through Prod::emit_code; otherwise the codes as
// kCodeTake / kCodeDrop / kCodeNever, each tile's taken count in its
// kTileTaken word).  Prod as for classify (a copy that writes no output from
// keys()).
template <class Prod>
__device__ uint32_t split_exact(const Prod& p, SpResolveShared& sh, const Layout& lay, const SelCtx& c, int32_t k,
                                int32_t* tiles, __amdgpu_buffer_rsrc_t codes) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  const int32_t ntile = (c.n + kSpTile - 1) / kSpTile;
  const int32_t per = (ntile + kSpWaves - 1) / kSpWaves;
  const int32_t w0 = __builtin_amdgcn_readfirstlane(min(wave * per, ntile));
  const int32_t w1 = __builtin_amdgcn_readfirstlane(min(w0 + per, ntile));
  uint32_t prefix = 0u;
  int32_t rem = k;
#pragma unroll 1
  for (int level = 0; level < 3; ++level) {
    const int shift = level == 0 ? 21 : level == 1 ? 10 : 0;
    const uint32_t mask = level == 2 ? 1023u : 2047u;
    const int pshift = level == 1 ? 21 : 10;
    for (int b = threadIdx.x; b < 2048; b += kSpThreads) sh.hist[b] = 0u;
    __syncthreads();
    FrameWin win;
    if (p.needs_class && w0 < w1) win.init(lay, c.seq, c.s0 + w0 * kSpTile);
    for (int32_t t = w0; t < w1; ++t) {
      uint32_t key[4];
      sp_tile_keys(p, win, c, t, key);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (key[e] != kSelNever && (level == 0 || (key[e] >> pshift) == (prefix >> pshift)))
          atomicAdd(&sh.hist[(key[e] >> shift) & mask], 1u);
    }
    __syncthreads();
    sp_pivot(sh.hist, rem, sh.wtot, sh.piv);
    prefix |= uint32_t(sh.piv[0]) << shift;
    rem = sh.piv[1];
    __syncthreads();
  }
  const uint32_t T = prefix;
  const int32_t need = rem;
  // keys equal to T per wave, then the waves' exclusive prefix
  int32_t eq = 0;
  {
    FrameWin win;
    if (p.needs_class && w0 < w1) win.init(lay, c.seq, c.s0 + w0 * kSpTile);
    for (int32_t t = w0; t < w1; ++t) {
      uint32_t key[4];
      sp_tile_keys(p, win, c, t, key);
#pragma unroll
      for (int e = 0; e < 4; ++e) eq += key[e] == T ? 1 : 0;
    }
  }
  eq = wave_sum(eq);
  if (lane == 0) sh.weq[wave] = eq;
  __syncthreads();
  int32_t eq_rank = 0;
  for (int w = 0; w < wave; ++w) eq_rank += sh.weq[w];
  // ranking walk: outputs (or codes and tile counts)
  FrameWin win;
  if (p.needs_class && w0 < w1) win.init(lay, c.seq, c.s0 + w0 * kSpTile);
  for (int32_t t = w0; t < w1; ++t) {
    uint32_t key[4];
    sp_tile_keys(p, win, c, t, key);
    int32_t taken = 0;
    uint32_t packed = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int32_t i = t * kSpTile + 64 * e + lane;
      const bool less = key[e] < T, tie = key[e] == T;
      const uint64_t beq = __ballot(tie);
      const bool take = less || (tie && eq_rank + __popcll(beq & below) < need);
      eq_rank += __popcll(beq);
      taken += __popcll(__ballot(take));
      if (Prod::kDirect) {
        if (i < c.n) p.emit_code(i, key[e] == kSelNever, take, 0);
      } else {
        packed |= (key[e] == kSelNever ? kCodeNever : take ? kCodeTake : kCodeDrop) << (8 * e);
      }
    }
    if (!Prod::kDirect) {
      __builtin_amdgcn_raw_buffer_store_b32(packed, codes, t * kSpTile + 4 * lane, 0, 0);
      if (lane == 0) tiles[size_t(t) * kTileWords + kTileTaken] = taken;
    }
  }
  return T;
}

// Resolve of one segment.  OFFSETS: write each tile's output offset (for a
// ranked list).  pe: the producer with no per-token output from keys() (the
// candidates' and ties' direct outputs go through pe.emit_code).  Returns T
// (valid for the modes that select) and sets *mode.
template <bool OFFSETS, class Prod>
__device__ uint32_t split_resolve(const Prod& pe, SpResolveShared& sh, const SelPlan& s, const Layout& lay,
                                  const SelCtx& c, int32_t* mode_out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int32_t* st = sp_state(s, lay);
  const uint32_t lo = uint32_t(st[kSpLo]), hi = uint32_t(st[kSpHi]);
  const int32_t k = st[kSpK];
  const int32_t count = st[kSpCount];
  int32_t mode = st[kSpMode];
  int32_t* tiles = sp_tiles(s, lay, c);
  int32_t cap;
  const uint2* cands = sp_cands(s, lay, c, &cap);
  const __amdgpu_buffer_rsrc_t codes = sp_codes(s, lay, c);
  const int32_t ntile = (c.n + kSpTile - 1) / kSpTile;
  const bool lds_tiles = ntile <= kSpLdsTiles;
  if (mode == kModeNone) {
    *mode_out = mode;
    return 0u;
  }
  if (mode == kModeAll) {  // every selectable token taken; T is the largest key
    uint32_t m = 0u;
    for (int32_t t = threadIdx.x; t < ntile; t += kSpThreads) {
      if (OFFSETS) tiles[size_t(t) * kTileWords + kTileOut] = t * kSpTile;
      m = max(m, uint32_t(tiles[size_t(t) * kTileWords + kTileMax]));
    }
    m = sp_wave_max(m);
    if (threadIdx.x == 0) sh.sum[0] = 0;
    __syncthreads();
    if (lane == 0) atomicMax(reinterpret_cast<uint32_t*>(&sh.sum[0]), m);
    __syncthreads();
    *mode_out = mode;
    return uint32_t(sh.sum[0]) - 1u;
  }
  // the candidate list's first batch, loaded while the totals are summed
  uint2 v[kSpPerThread];
  const int32_t nlist = min(count, cap);
  auto reload = [&](int32_t i0) {
#pragma unroll
    for (int e = 0; e < kSpPerThread; ++e) {
      const int32_t i = i0 + e * kSpThreads + int32_t(threadIdx.x);
      v[e] = i < nlist ? cands[i] : make_uint2(kSelNever, 0u);
    }
  };
  const bool one = nlist <= kSpBatch;
  reload(0);
  // totals of the four codes (keys below lo, equal to lo, strictly between,
  // equal to hi), summed by classify into the state words
  const int32_t N1 = st[kSpEqLo];
  const int32_t N0 = st[kSpLe] - N1;
  const int32_t N2 = count;
  const int32_t N3 = st[kSpEqHi];
  if (s.split_exact || k <= N0) mode = kModeExact;
  else if (k <= N0 + N1) mode = kModeTieLo;
  else if (k <= N0 + N1 + N2) mode = count <= cap ? kModeMid : kModeExact;
  else if (k <= N0 + N1 + N2 + N3) mode = (Prod::kDirect && count > cap) ? kModeExact : kModeTieHi;
  else mode = kModeExact;

  uint32_t T = 0u;
  int32_t need = 0, cut = c.n, tstar = -1, tie_before = 0;
  if (mode == kModeMid) {
    int32_t m_eq = 0;
    T = sp_cand_select([](const uint2& x) { return x.x; }, reload, v, count, one, k - N0 - N1, lo + 1u, hi - 1u, sh,
                       &need, &m_eq);
    if (need < m_eq) {  // not every candidate equal to T is taken: cut at the need-th one in index order
      if (m_eq <= kSpTieMax) cut = sp_tie_cut(reload, v, count, one, T, need, m_eq, c.n, sh);
      else mode = kModeExact;  // (streamed below)
    }
  }
  if (mode == kModeExact) {
    T = split_exact(pe, sh, lay, c, k, tiles, codes);
  } else if (mode == kModeMid) {
    if (OFFSETS && lds_tiles) {
      for (int32_t t = threadIdx.x; t < ntile; t += kSpThreads) sh.tcount[t] = 0;
      __syncthreads();
    }
    for (int32_t i0 = 0; i0 < count; i0 += kSpBatch) {
      if (!one) reload(i0);
#pragma unroll
      for (int e = 0; e < kSpPerThread; ++e) {
        if (v[e].x == kSelNever) continue;
        const bool take = v[e].x < T || (v[e].x == T && int32_t(v[e].y) <= cut);
        if (Prod::kDirect) {
          if (take) pe.emit_code(int32_t(v[e].y), false, true, 0);
        } else {
          __builtin_amdgcn_raw_buffer_store_b8(uint8_t(take ? kCodeTake : kCodeDrop), codes,
                                               sp_code_off(int32_t(v[e].y)), 0, 0);
        }
        if (OFFSETS && take) {
          const int32_t t = int32_t(v[e].y / kSpTile);
          if (lds_tiles) atomicAdd(&sh.tcount[t], 1);
          else atomicAdd(&tiles[size_t(t) * kTileWords + kTileTaken], 1);
        }
      }
    }
  } else {  // a tie at lo or at hi: the first `need` tied tokens in index order
    const int word = mode == kModeTieLo ? kTileEqLo : kTileEqHi;
    T = mode == kModeTieLo ? lo : hi;
    need = mode == kModeTieLo ? k - N0 : k - (N0 + N1 + N2);
    if (threadIdx.x == 0) {
      sh.found[0] = -1;
      sh.found[1] = 0;
      sh.cut = c.n - 1;
    }
    __syncthreads();
    int32_t run = 0;
    for (int32_t b0 = 0; b0 < ntile; b0 += kSpThreads) {
      const int32_t t = b0 + int32_t(threadIdx.x);
      const int32_t x = t < ntile ? tiles[size_t(t) * kTileWords + word] : 0;
      int32_t total;
      const int32_t incl = sp_block_inscan(x, sh.wtot, &total) + run;
      if (t < ntile && incl >= need && incl - x < need) {
        sh.found[0] = t;
        sh.found[1] = incl - x;
      }
      run += total;
      __syncthreads();
      if (sh.found[0] >= 0) break;
    }
    tstar = sh.found[0];
    tie_before = sh.found[1];
    if (wave == 0 && tstar >= 0) {  // the cut: the (need - tie_before)-th tied token of tile tstar
      FrameWin win;
      if (pe.needs_class) win.init(lay, c.seq, c.s0 + tstar * kSpTile);
      uint32_t key[4];
      sp_tile_keys(pe, win, c, tstar, key);
      int32_t r = need - tie_before;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint64_t m = __ballot(key[e] == T);
        const int32_t pc = __popcll(m);
        if (r > 0 && r <= pc && key[e] == T && __popcll(m & below) == r - 1) sh.cut = tstar * kSpTile + 64 * e + lane;
        r -= pc;
      }
    }
    __syncthreads();
    cut = sh.cut;
    if (Prod::kDirect) {
      // the open tokens of a tie: at hi the candidates are all taken, then the
      // tied tokens up to the cut (classify wrote 1 at lo and 0 at hi)
      if (mode == kModeTieHi)
        for (int32_t i0 = 0; i0 < count; i0 += kSpBatch) {
          if (!one) reload(i0);
#pragma unroll
          for (int e = 0; e < kSpPerThread; ++e)
            if (v[e].x != kSelNever) pe.emit_code(int32_t(v[e].y), false, true, 0);
        }
      // tiles holding tied tokens, each walked by one wave in increasing order
      FrameWin win;
      bool started = false;
      for (int32_t t = wave; t < ntile; t += kSpWaves) {
        const bool side = mode == kModeTieLo ? t >= tstar : t <= tstar;
        if (!side || tiles[size_t(t) * kTileWords + word] == 0) continue;
        if (pe.needs_class && !started) win.init(lay, c.seq, c.s0 + t * kSpTile);
        started = true;
        uint32_t key[4];
        sp_tile_keys(pe, win, c, t, key);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int32_t i = t * kSpTile + 64 * e + lane;
          if (key[e] == T && i < c.n) pe.emit_code(i, false, i <= cut, 0);
        }
      }
    }
  }
  if (OFFSETS) {
    // the counts written above (stores and atomics of this work-group) are
    // complete before any thread reads them back past the vector L1
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    int32_t run = 0;
    for (int32_t b0 = 0; b0 < ntile; b0 += kSpThreads) {
      const int32_t t = b0 + int32_t(threadIdx.x);
      int32_t x = 0;
      if (t < ntile) {
        const int32_t* r = tiles + size_t(t) * kTileWords;
        if (mode == kModeExact) {
          x = sp_load_agent(r + kTileTaken);
        } else if (mode == kModeMid) {
          x = r[kTileLess] + r[kTileEqLo] + (lds_tiles ? sh.tcount[t] : sp_load_agent(r + kTileTaken));
        } else {
          const int word = mode == kModeTieLo ? kTileEqLo : kTileEqHi;
          x = mode == kModeTieLo ? r[kTileLess] : r[kTileLess] + r[kTileEqLo] + r[kTileMid];
          x += t < tstar ? r[word] : t == tstar ? need - tie_before : 0;
        }
      }
      int32_t total;
      const int32_t incl = sp_block_inscan(x, sh.wtot, &total) + run;
      if (t < ntile) tiles[size_t(t) * kTileWords + kTileOut] = incl - x;
      run += total;
    }
  }
  if (threadIdx.x == 0) {
    st[kSpMode] = mode;
    st[kSpT] = int32_t(T);
    st[kSpCut] = cut;
    st[kSpNeed] = need;
  }
  *mode_out = mode;
  return T;
}

// ---------------------------------------------------------------------------
// emit: a ranked list from the codes (grid (parts, seqs, units),
// kSpPassThreads threads)
// ---------------------------------------------------------------------------

// Prod provides void emit_code(int32_t i, bool never, bool take, int32_t pos)
// for every token of the part (pos: its rank among the segment's taken
// tokens).  A wave loads the codes of kSpEmitBatch of its tiles at once.
template <class Prod>
__device__ void split_emit(const Prod& p, const SelPlan& s, const Layout& lay, const SelCtx& c) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  const int32_t* st = sp_state(s, lay);
  const int32_t mode = st[kSpMode];
  if (mode == kModeNone) return;
  const int32_t cut = st[kSpCut];
  // codes below `lim` are taken; a tie code `tc` is taken up to the cut
  const uint32_t lim = mode == kModeTieLo ? 1u : mode == kModeMid ? 2u : mode == kModeTieHi ? 3u : 0u;
  const uint32_t tc = mode == kModeTieLo ? kCodeEqLo : mode == kModeTieHi ? kCodeEqHi : 0xffu;
  int32_t t0, t1;
  sp_part_tiles(c.n, s.split_parts, c.part, &t0, &t1);
  const int32_t* tiles = sp_tiles(s, lay, c);
  const __amdgpu_buffer_rsrc_t codes = sp_codes(s, lay, c);
  const int32_t tw = t0 + wave;
  const int32_t nt = tw < t1 ? (t1 - tw + kSpPassWaves - 1) / kSpPassWaves : 0;
  for (int32_t j0 = 0; j0 < nt; j0 += kSpEmitBatch) {
    uint32_t packed[kSpEmitBatch];
    int32_t out[kSpEmitBatch];
#pragma unroll
    for (int j = 0; j < kSpEmitBatch; ++j) {
      const int32_t t = tw + kSpPassWaves * (j0 + j);
      const bool ok = j0 + j < nt;
      packed[j] = ok ? __builtin_amdgcn_raw_buffer_load_b32(codes, t * kSpTile + 4 * lane, 0, 0) : 0u;
      out[j] = ok ? tiles[size_t(t) * kTileWords + kTileOut] : 0;
    }
#pragma unroll
    for (int j = 0; j < kSpEmitBatch; ++j) {
      if (j0 + j >= nt) break;
      const int32_t t = tw + kSpPassWaves * (j0 + j);
      int32_t o = out[j];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int32_t i = t * kSpTile + 64 * e + lane;
        const uint32_t code = (packed[j] >> (8 * e)) & 255u;
        const bool take = i < c.n && (code == kCodeTake || code < lim || (code == tc && i <= cut));
        const uint64_t m = __ballot(take);
        if (take) p.emit_code(i, false, true, o + __popcll(m & below));
        o += __popcll(m);
      }
    }
  }
}

// The frames of sequence seq; with LDS, their ranges copied to fs / fe (the
// caller synchronises before using them).
template <bool LDS>
__device__ inline SeqFrames<LDS> sp_frames(int32_t* fs, int32_t* fe, const Layout& lay, int32_t seq) {
  SeqFrames<LDS> fr;
  fr.meta = lay.frame_meta;
  fr.fs = fs;
  fr.fe = fe;
  fr.f0 = lay.cu_frames[seq];
  fr.nf = lay.cu_frames[seq + 1] - fr.f0;
  if constexpr (LDS) {
    for (int32_t f = threadIdx.x; f < fr.nf; f += blockDim.x) {
      const int32_t* m = lay.frame_meta + 3 * (fr.f0 + f);
      fs[f] = m[0];
      fe[f] = m[0] + m[1] * m[2];
    }
  }
  return fr;
}

// The launches: sample and resolve over (1, sequences, units), classify and
// (with an emit kernel: ranked lists) emit over (split_parts, sequences,
// units).
//
// The classify and emit grids are sized to whole rounds of the work-groups
// the GPU holds at once (the classify kernel's occupancy on 256 CUs), so that
// no last round runs on a fraction of the chip: the parts per segment are a
// round's work-groups over the segments, in as many rounds as keep a
// work-group to at most 64 tiles.  Without an occupancy figure the plan's
// part count (32 tiles per work-group) stays.
template <class Args>
hipError_t launch_split(void (*sample)(Args), void (*classify)(Args), void (*resolve)(Args), void (*emit)(Args),
                        const Args& a_in, const Layout& lay, hipStream_t stream) {
  if (lay.n_units == 0 || lay.n_seqs == 0) return hipSuccess;
  // Work-groups of the classify kernel per CU (-1: unknown), queried on the
  // first call; a function-local static is initialised once even when
  // several host threads make that first call together.
  static const int occupancy = [classify]() {
    int b = 0;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, classify, kSpPassThreads, 0) == hipSuccess && b > 0 ? b
                                                                                                              : -1;
  }();
  Args a = a_in;
  SelPlan& s = a.sel;
  if (occupancy > 0) {
    const int64_t segs = int64_t(lay.n_units) * lay.n_seqs;
    const int64_t per_round = std::max<int64_t>(1, int64_t(256) * occupancy / segs);
    const int64_t tiles = std::max<int64_t>(1, s.split_tiles);
    const int64_t rounds = std::max<int64_t>(1, (tiles + 64 * per_round - 1) / (64 * per_round));
    s.split_parts = int32_t(std::min<int64_t>(rounds * per_round, tiles));
  }
  const dim3 seg_grid(1, lay.n_seqs, lay.n_units), pass_grid(s.split_parts, lay.n_seqs, lay.n_units);
  hipLaunchKernelGGL(sample, seg_grid, dim3(kSpThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(classify, pass_grid, dim3(kSpPassThreads), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(resolve, seg_grid, dim3(kSpThreads), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess || !emit) return e;
  hipLaunchKernelGGL(emit, pass_grid, dim3(kSpPassThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
