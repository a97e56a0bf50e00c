// Decode attention over a KV cache: the decoding phase of the problem setup,
// which attends each new query over the cached keys and values -- the full
// prefill cache, or the compressed K', V' the compression procedure returns:
//   out_g = sum_j softmax_j(q_g . k_j / sqrt(d)) v_j
// for every layer, sequence and query head g, over the sequence's rows of the
// cache (the decode query comes after all of them: no mask).
//
// Split-K flash decoding.  A work-group takes one chunk of a sequence's rows
// of one kv head; its four waves take 16-row sub-tiles in turn:
//   S^T = K Q^T   v_mfma_f32_16x16x32_bf16, cached rows as the A operand read
//                 straight from HBM, the GQA group's queries (G <= 16, zero
//                 padded) resident as the B operand;
//   online softmax per head in fp32 (log2 units);
//   O += P V      v_mfma_f32_16x16x4_f32, which takes one cached row per lane
//                 and k-step: V rows load straight from HBM as 16-byte pieces
//                 with no transpose, and P stays fp32.
// Each wave keeps (max, sum, O) per head; the waves are merged in LDS and the
// chunk's partial is written; a combine kernel merges the chunks of each
// sequence.  The pass streams K and V once: HBM-bound.
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr float kScale2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
constexpr int kDecWaves = 4;
constexpr int kDecHeads = 16;  // query heads of a kv head, padded
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// 16 bytes of a cached row, read once by the whole call: a non-temporal load
// (streaming reads reach ~6.2 TB/s this way against ~5.6 with the default
// policy).
__device__ inline uint4 load_row16(const uint16_t* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

struct RowChunk {
  int32_t seq, row0, c0, c1, gchunk;  // c0, c1: row range local to the sequence
};

// Work-group x index -> (sequence, row range) for a fixed chunk length.
__device__ inline RowChunk locate_rows(const DecodeArgs& a, int32_t gchunk) {
  RowChunk r{-1, 0, 0, 0, gchunk};
  int32_t acc = 0;
  for (int32_t s = 0; s < a.lay.n_seqs; ++s) {
    const int32_t lo = a.cu_rows[s], hi = a.cu_rows[s + 1];
    const int32_t n = (hi - lo + a.chunk - 1) / a.chunk;
    if (gchunk < acc + n) {
      r.seq = s;
      r.row0 = lo;
      r.c0 = (gchunk - acc) * a.chunk;
      r.c1 = min(r.c0 + a.chunk, hi - lo);
      return r;
    }
    acc += n;
  }
  return r;
}

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// One chunk: per-head (max, sum) and unnormalised O of the chunk's rows.
__global__ __launch_bounds__(kDecWaves * 64) void decode_chunk_kernel(DecodeArgs a) {
  __shared__ float sm_m[kDecWaves][kDecHeads], sm_l[kDecWaves][kDecHeads];
  __shared__ float sm_o[kDecWaves][kDecHeads][kHeadDim];
  const int unit = blockIdx.y;
  const RowChunk rc = locate_rows(a, blockIdx.x);
  if (rc.seq < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int layer = unit / a.lay.n_kv_heads, kv = unit % a.lay.n_kv_heads;
  const int head = lane & 15, quad = lane >> 4;

  // Queries as the B operand: lane supplies head `head`, dims 32 kk + 8 quad .. +7.
  bf16x8_t qb[4];
  {
    const uint16_t* qrow =
        a.q + ((size_t(layer) * a.lay.n_seqs + rc.seq) * a.n_q_heads + size_t(kv) * a.group + head) * kHeadDim;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (head < a.group) v = *reinterpret_cast<const uint4*>(qrow + kk * 32 + quad * 8);
      qb[kk] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
  const size_t base = (size_t(unit) * a.total_rows + rc.row0) * kHeadDim;
  const uint16_t* krows = a.k + base;
  const uint16_t* vrows = a.v + base;

  float m_run = -INFINITY;  // per head `head` (the same in its four lanes)
  float l_run = 0.0f;       // this lane's part of the head's sum
  f32x4_t o[8];             // O[head 4 quad + r][dim 8 (lane & 15) + db]
#pragma unroll
  for (int db = 0; db < 8; ++db) o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Sub-tile rows j0 .. j0+15: K row j0 + (lane & 15) (A operand, dims 32 kk +
  // 8 quad ..) and V rows j0 + 4 quad + i, dims 8 (lane & 15) .. +7.  Rows past
  // the chunk read its last row and are masked.
  uint4 kx[4], vx[4];
  auto load = [&](int32_t j0) {
    const int32_t jk = min(j0 + (lane & 15), rc.c1 - 1);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      kx[kk] = load_row16(krows + size_t(jk) * kHeadDim + kk * 32 + quad * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t jv = min(j0 + 4 * quad + i, rc.c1 - 1);
      vx[i] = load_row16(vrows + size_t(jv) * kHeadDim + (lane & 15) * 8);
    }
  };
  int32_t j0 = rc.c0 + 16 * wave;
  if (j0 < rc.c1) load(j0);
  for (; j0 < rc.c1; j0 += 16 * kDecWaves) {
    const uint4 kc[4] = {kx[0], kx[1], kx[2], kx[3]};
    const uint4 vc[4] = {vx[0], vx[1], vx[2], vx[3]};
    if (j0 + 16 * kDecWaves < rc.c1) load(j0 + 16 * kDecWaves);  // next sub-tile in flight

    // S^T: lane holds head `head`, rows j0 + 4 quad + i.
    f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kc[kk]), qb[kk], s, 0, 0, 0);
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = j0 + 4 * quad + i < rc.c1 ? s[i] * kScale2 : -INFINITY;
    float mt = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    // Row j0 is in the chunk, so every head's tile maximum is finite.
    const float m_new = fmaxf(m_run, mt);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(x[i] - m_new);
    l_run = l_run * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    m_run = m_new;
    // O rows are heads 4 quad + r; their factors live in lanes 4 quad + r.
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ar = __shfl(alpha, 4 * quad + r);
#pragma unroll
      for (int db = 0; db < 8; ++db) o[db][r] *= ar;
    }
    // O += P V: k-step i pairs lane (head, quad) with row j0 + 4 quad + i.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t w[4] = {vc[i].x, vc[i].y, vc[i].z, vc[i].w};
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const float b = (db & 1) ? bf16_hi(w[db >> 1]) : bf16_lo(w[db >> 1]);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(p[i], b, o[db], 0, 0, 0);
      }
    }
  }

  // The head's sum over its four lanes; the wave's state to LDS.
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (lane < kDecHeads) {
    sm_m[wave][lane] = m_run;
    sm_l[wave][lane] = l_run;
  }
#pragma unroll
  for (int db = 0; db < 8; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) sm_o[wave][4 * quad + r][(lane & 15) * 8 + db] = o[db][r];
  __syncthreads();

  // Merge the waves (a wave without rows has max -inf and weighs nothing).
  float* pm = a.pm + (size_t(unit) * a.total_chunks + rc.gchunk) * kDecHeads;
  float* pl = a.pl + (size_t(unit) * a.total_chunks + rc.gchunk) * kDecHeads;
  float* po = a.po + (size_t(unit) * a.total_chunks + rc.gchunk) * kDecHeads * kHeadDim;
  for (int e = threadIdx.x; e < a.group * kHeadDim; e += kDecWaves * 64) {
    const int h = e / kHeadDim, dim = e % kHeadDim;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, sm_m[w][h]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float wt = sm_m[w][h] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(sm_m[w][h] - M);
      L += wt * sm_l[w][h];
      O += wt * sm_o[w][h][dim];
    }
    po[h * kHeadDim + dim] = O;
    if (dim == 0) {
      pm[h] = M;
      pl[h] = L;
    }
  }
}

// Per (unit, sequence, query head): merge the chunks, out = O / L (0 for a
// sequence without rows).  One output dimension per thread.  The partials of
// kCombineBatch chunks are loaded before any of them is merged, so a batch
// costs one memory latency; the batch is weighed against its maximum (a chunk
// that saw no row of the sequence has max -inf and weighs nothing) and merged
// into the running (M, L, O).
constexpr int kCombineBatch = 16;

__global__ __launch_bounds__(kHeadDim) void decode_combine_kernel(DecodeArgs a) {
  const int32_t s = blockIdx.x;
  const int unit = blockIdx.y, h = blockIdx.z;
  const int dim = threadIdx.x;
  const int layer = unit / a.lay.n_kv_heads, kv = unit % a.lay.n_kv_heads;
  int32_t first = 0;
  for (int32_t t = 0; t < s; ++t) first += (a.cu_rows[t + 1] - a.cu_rows[t] + a.chunk - 1) / a.chunk;
  const int32_t nch = (a.cu_rows[s + 1] - a.cu_rows[s] + a.chunk - 1) / a.chunk;
  const size_t c0 = size_t(unit) * a.total_chunks + first;
  float M = -INFINITY, L = 0.0f, O = 0.0f;
  for (int32_t b0 = 0; b0 < nch; b0 += kCombineBatch) {
    float m[kCombineBatch], l[kCombineBatch], o[kCombineBatch];
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) {
      // slots past the sequence's last chunk re-read that chunk and weigh nothing
      const size_t ch = (c0 + size_t(min(b0 + i, nch - 1))) * kDecHeads + h;
      const float mv = a.pm[ch];
      l[i] = a.pl[ch];
      o[i] = a.po[ch * kHeadDim + dim];
      m[i] = b0 + i < nch ? mv : -INFINITY;
    }
    float mx = M;
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) mx = fmaxf(mx, m[i]);
    if (mx == -INFINITY) continue;  // no chunk so far saw a row of the sequence
    const float sa = __builtin_amdgcn_exp2f(M - mx);  // 0 while M is still -inf
    L *= sa;
    O *= sa;
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) {
      const float w = m[i] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m[i] - mx);
      L += w * l[i];
      O += w * o[i];
    }
    M = mx;
  }
  a.out[((size_t(layer) * a.lay.n_seqs + s) * a.n_q_heads + size_t(kv) * a.group + h) * kHeadDim + dim] =
      L > 0.0f ? O / L : 0.0f;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  if (a.total_chunks > 0) {
    hipLaunchKernelGGL(decode_chunk_kernel, dim3(a.total_chunks, a.lay.n_units), dim3(kDecWaves * 64), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(decode_combine_kernel, dim3(a.lay.n_seqs, a.lay.n_units, a.group), dim3(kHeadDim), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
