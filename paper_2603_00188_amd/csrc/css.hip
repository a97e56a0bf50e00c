// Component-centric Spatial Saliency (Eq. css_calc of the paper):
//   H_{u,v} = mean over the in-grid Moore neighbours n of cos(h_{u,v}, h_n),
//   Phi = 1 - H  (0 when a frame is 1x1; 0 on text tokens).
//
// One wave sweeps a vertical strip of a frame row by row.  A strip is 16
// loaded columns: 14 output columns plus one halo column on each side.  Four
// lanes share a cell, each holding 32 of the 128 dimensions, so a dot product
// is 16 v_dot2 per lane and a two-step quad reduction.
//
// Each unordered neighbour pair is evaluated once: a cell computes only its
// forward cosines E (r, c+1), S (r+1, c), SE (r+1, c+1) and SW (r+1, c-1).
// Row r's mean combines its own forward cosines, its west neighbour's E, and
// the previous row's S / SE / SW carried in registers.
//
// Rows stream into a four-slot LDS ring by direct memory->LDS DMA, two rows
// ahead of the row being combined, so every key is read from HBM once per
// strip.  The strips of one frame are given to work-groups that land on the
// same XCD, where the halo columns hit the shared L2.
//
// With the TSG gate given (GATED), a token whose gate is 0 gets Phi = 0 (its
// saliency is multiplied away by M = 0 in Eq. modal_scoring), and a strip row
// whose cosines no admitted cell of that row or the next needs skips them
// (the row is still loaded: its keys are the neighbours of the rows around
// it).  Each lane's gate byte is loaded three rows ahead, right after the
// row's DMA, so the loads complete in the same order as the ring rows.
//
// The neighbourhood-size ablation widens the window to k x k, k = 2 KR + 1 in
// {5, 7, 9} (css_wide_kernel): H = mean over the in-grid cells of the square
// other than the centre.  There the cosines form a small dense contraction,
// which runs on the matrix cores: a wave owns a 4-row x 16-column output tile
// whose 64 keys stay in VGPRs as MFMA A operands, and walks the 4 + 2 KR
// neighbour rows.  Each neighbour row's 16 + 2 KR columns (two 16-key B
// blocks) are multiplied with every output row within KR of it; a per-lane
// mask keeps the products with |dc| <= KR, scales them by the neighbour's
// inverse norm and adds them in the accumulator lanes, and one 16-lane
// reduction per output finishes the sum.  Halo rows shared by neighbouring
// tiles are re-read through L2 (the tiles of one frame go to one XCD).
#include "stlite_internal.h"
#include "tile_lds.h"

namespace stlite {
namespace {

constexpr int kStripCells = 16;  // loaded columns per strip (one per lane quad)
constexpr int kStripOut = 14;    // output columns per strip
constexpr int kRowElems = kStripCells * kHeadDim;
constexpr int kRowLoads = kStripCells * kHeadDim * 2 / (64 * 16);  // wave-loads of 16 B per lane: 4

// The 16-byte chunk ch (dims 8ch .. 8ch+7) of loaded cell g sits at slot
// ch ^ 4 (g & 1): lanes 0..7 of a b128 read then cover all 32 banks.
__device__ inline int chunk_slot(int g, int ch) { return ch ^ ((g & 1) << 2); }

// DMA of one strip row (16 cells, column-clamped) into `dst`.
__device__ inline void row_dma(const uint16_t* kframe, int32_t row, int32_t c0, int32_t C, uint16_t* dst) {
  const int lane = threadIdx.x & 63;
  // The slot being refilled was last read two steps ago; make sure those LDS
  // reads have completed before the DMA can land.
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  // A buffer load into LDS over the frame row: tracked by the vector-memory
  // counter only, so the ring reads keep exact lgkmcnt waits.
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(kframe + size_t(row) * C * kHeadDim), 0, C * (kHeadDim * 2), kBufferFlags);
#pragma unroll
  for (int m = 0; m < kRowLoads; ++m) {
    const int g = 4 * m + (lane >> 4);
    const int slot = lane & 15;
    const int ch = chunk_slot(g, slot);  // the mapping is its own inverse
    const int32_t col = min(max(c0 - 1 + g, 0), C - 1);
    // The LDS address goes through an opaque copy, so the compiler does not
    // tie the DMA to the ring array and add its own (full) vmcnt waits before
    // the ring is read; the kernel waits for exactly the rows it needs.
    uint32_t lds = uint32_t(reinterpret_cast<uintptr_t>(dst + 4 * m * kHeadDim));
    asm volatile("" : "+s"(lds));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t)(uintptr_t)lds, 16,
                                             uint32_t(col) * (kHeadDim * 2) + uint32_t(ch) * 16u, 0, 0, 0);
  }
}

// Lane (g, s) holds chunks s, s+4, s+8, s+12 of cell g.
struct Slice {
  uint4 c[4];
};

__device__ inline Slice read_slice(const uint16_t* row, int g, int s) {
  Slice x;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    x.c[j] = *reinterpret_cast<const uint4*>(row + g * kHeadDim + chunk_slot(g, 4 * j + s) * 8);
  return x;
}

__device__ inline float dot_slice(const Slice& a, const Slice& b) {
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t wa[4] = {a.c[j].x, a.c[j].y, a.c[j].z, a.c[j].w};
    const uint32_t wb[4] = {b.c[j].x, b.c[j].y, b.c[j].z, b.c[j].w};
#pragma unroll
    for (int i = 0; i < 4; ++i)
      s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, wa[i]), __builtin_bit_cast(bf16x2_t, wb[i]), s,
                                          false);
  }
  return s;
}

// Sum over the four lanes of a quad (lanes 4g .. 4g+3).
__device__ inline float quad_sum(float x) {
  x += __shfl_xor(x, 1);
  x += __shfl_xor(x, 2);
  return x;
}

// 1/||k|| from ||k||^2 (0 for a zero key).  v_rsq_f32 (1 ulp) covers every
// normal square norm; the exactly rounded form is kept for tiny ones.
__device__ inline float inv_norm(float ss) {
  float r = __builtin_amdgcn_rsqf(ss);
  if (!(ss >= 0x1p-100f)) r = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
  return r;
}

template <bool GATED>
__global__ __launch_bounds__(64) void css_kernel(CssArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ring0[kRowElems], ring1[kRowElems], ring2[kRowElems],
      ring3[kRowElems];
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  // XCD-aware order: work-groups i, i + 8, i + 16, ... share an XCD, so they
  // take consecutive strips (the grid width is a multiple of 8).
  const int32_t per_xcd = int32_t(gridDim.x) >> 3;
  const int32_t logical = int32_t(blockIdx.x & 7) * per_xcd + int32_t(blockIdx.x >> 3);
  const int32_t f = logical / a.strips, strip = logical - f * a.strips;
  if (f >= lay.n_frames) return;
  const int32_t off = lay.frame_meta[3 * f], R = lay.frame_meta[3 * f + 1], C = lay.frame_meta[3 * f + 2];
  const int32_t c0 = strip * kStripOut;
  if (c0 >= C) return;

  const int lane = threadIdx.x & 63, g = lane >> 2, s = lane & 3;
  const int32_t col = c0 - 1 + g;
  const bool out_lane = g >= 1 && g <= kStripOut && col < C;
  const bool has_w = col >= 1, has_e = col + 1 < C;
  const int32_t ncols = 1 + (col > 0 ? 1 : 0) + (col < C - 1 ? 1 : 0);
  const uint16_t* kframe = a.k + (size_t(unit) * lay.total_tokens + off) * kHeadDim;
  // Phi of the frame through a buffer resource: lanes without an output store
  // to an offset past the end, which the hardware drops, so the store needs no
  // branch (and the number of memory operations per step stays fixed).
  const uint32_t frame_bytes = uint32_t(R) * uint32_t(C) * 4u;
  const __amdgpu_buffer_rsrc_t phi_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(a.phi + size_t(unit) * lay.total_tokens + off, 0, frame_bytes, kBufferFlags);
  const int ge = min(g + 1, kStripCells - 1), gw = max(g - 1, 0);
  // The gate bytes of the frame (GATED): lanes without an output read an
  // offset past the end, which returns 0.
  const __amdgpu_buffer_rsrc_t gate_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(GATED ? a.gate + size_t(unit) * lay.total_tokens + off : nullptr), 0,
      GATED ? uint32_t(R) * uint32_t(C) : 0u, kBufferFlags);
  const uint32_t gate_none = uint32_t(R) * uint32_t(C);
  auto gate_load = [&](int32_t row) -> uint32_t {
    return __builtin_amdgcn_raw_buffer_load_b8(gate_rsrc, out_lane ? uint32_t(row * C + col) : gate_none, 0, 0);
  };
  // vector-memory operations per ring row: its DMA and, gated, the gate bytes
  constexpr int kPerRow = kRowLoads + (GATED ? 1 : 0);

  // Every step issues one row (rows past the end repeat row R-1 and hit L2),
  // so the number of loads in flight is the same on every path: 2 rows.
  uint32_t g0 = 1, g1 = 1, g2 = 1, g3 = 1;  // gates of rows r .. r+3 (GATED)
  row_dma(kframe, 0, c0, C, ring0);
  if (GATED) g0 = gate_load(0);
  row_dma(kframe, min(1, R - 1), c0, C, ring1);
  if (GATED) g1 = gate_load(min(1, R - 1));
  row_dma(kframe, min(2, R - 1), c0, C, ring2);
  if (GATED) g2 = gate_load(min(2, R - 1));

  // Row 0: own slice and inverse norm.
  wait_vmcnt<2 * kPerRow>();
  Slice own = read_slice(ring0, g, s);
  float rn_own = inv_norm(quad_sum(dot_slice(own, own)));
  float carry = 0.0f;  // sum of row r-1's cosines with (r, col)

  auto step = [&](int32_t r, uint16_t* cur, uint16_t* nxt, uint16_t* issue_dst) {
    const bool has_s = r + 1 < R;
    row_dma(kframe, min(r + 3, R - 1), c0, C, issue_dst);
    if (GATED) g3 = gate_load(min(r + 3, R - 1));
    wait_vmcnt<2 * kPerRow>();  // row r+1 (and its gate bytes) have landed
    // Row r+1 (on the last row the slot holds a repeat of row R-1; masked).
    const Slice down = read_slice(nxt, g, s);
    const float rn_down = inv_norm(quad_sum(dot_slice(down, down)));
    // The cosines of this step serve rows r and r+1: skip them when no cell
    // of either needs its Phi (wave-uniform).
    const bool need = r < R && (!GATED || __ballot(out_lane && (g0 | g1) != 0u) != 0);
    float H = 0.0f;
    if (need) {
      // East neighbour in this row; norms of the east cell come by shuffle.
      const Slice e = read_slice(cur, ge, s);
      const float dE = quad_sum(dot_slice(own, e));
      const float rnE = __shfl(rn_own, (ge << 2) | s);
      const float cE = has_e ? dE * rn_own * rnE : 0.0f;
      const Slice se = read_slice(nxt, ge, s);
      const Slice sw = read_slice(nxt, gw, s);
      const float dS = quad_sum(dot_slice(own, down));
      const float dSE = quad_sum(dot_slice(own, se));
      const float dSW = quad_sum(dot_slice(own, sw));
      const float rnSE = __shfl(rn_down, (ge << 2) | s);
      const float rnSW = __shfl(rn_down, (gw << 2) | s);
      const float cS = has_s ? dS * rn_own * rn_down : 0.0f;
      const float cSE = has_s && has_e ? dSE * rn_own * rnSE : 0.0f;
      const float cSW = has_s && has_w ? dSW * rn_own * rnSW : 0.0f;
      // Cosines owned by the west / east neighbours of this cell.
      const float cE_w = __shfl(cE, (gw << 2) | s);
      const float cSE_w = __shfl(cSE, (gw << 2) | s);
      const float cSW_e = __shfl(cSW, (ge << 2) | s);
      H = carry + cE + cS + cSE + cSW + (has_w ? cE_w : 0.0f);
      carry = cS + (has_w ? cSE_w : 0.0f) + (has_e ? cSW_e : 0.0f);
    } else {
      carry = 0.0f;  // row r+1 has no admitted cell either
    }
    const int32_t nrows = 1 + (r > 0 ? 1 : 0) + (has_s ? 1 : 0);
    const int32_t nn = nrows * ncols - 1;
    const bool store = r < R && out_lane && s == 0;
    const uint32_t byte_off = store ? uint32_t(r * C + col) * 4u : frame_bytes;
    const bool zero = nn <= 0 || (GATED && g0 == 0u);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(zero ? 0.0f : 1.0f - H * __builtin_amdgcn_rcpf(float(nn))),
                                          phi_rsrc, byte_off, 0, 0);
    own = down;
    rn_own = rn_down;
    g0 = g1;
    g1 = g2;
    g2 = g3;
  };

  // Row r lives in slot r % 4; unrolled by four so each slot is a distinct
  // array.  Steps past the last row only keep the load count uniform.
  for (int32_t r = 0; r < R; r += 4) {
    step(r, ring0, ring1, ring3);
    step(r + 1, ring1, ring2, ring0);
    step(r + 2, ring2, ring3, ring1);
    step(r + 3, ring3, ring0, ring2);
  }
  wait_vmcnt<0>();  // no DMA into LDS may outlive the work-group
}

constexpr int kWideRows = 4;   // output rows of a wave tile
constexpr int kWideCols = 16;  // output columns of a wave tile

__device__ inline float sumsq8(uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[j]), __builtin_bit_cast(bf16x2_t, w[j]), s, false);
  return s;
}

// Loads the MFMA operand fragments of key (row, col) of a frame: lane (n, q)
// holds dims 32 kk + 8 q .. 32 kk + 8 q + 7 for kk = 0..3, and returns the
// key's inverse norm (the same on the four lanes that share n).
__device__ inline float load_key_operand(const uint16_t* kframe, int32_t row, int32_t col, int32_t C, int q,
                                         bf16x8_t (&frag)[4]) {
  const uint16_t* src = kframe + (size_t(row) * C + col) * kHeadDim + q * 8;
  float ss = 0.0f;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const uint4 v = *reinterpret_cast<const uint4*>(src + kk * 32);
    ss += sumsq8(v);
    frag[kk] = __builtin_bit_cast(bf16x8_t, v);
  }
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  return inv_norm(ss);
}

// Grid: x = work-groups of four wave tiles, in XCD-aware order; a.strips is
// the largest number of 4 x 16 tiles of a frame; y = unit.
template <int KR>
__global__ __launch_bounds__(256) void css_wide_kernel(CssArgs a) {
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t per_xcd = int32_t(gridDim.x) >> 3;
  const int32_t logical = (int32_t(blockIdx.x & 7) * per_xcd + int32_t(blockIdx.x >> 3)) * 4 + wave;
  const int32_t f = logical / a.strips, t = logical - f * a.strips;
  if (f >= lay.n_frames) return;
  const int32_t off = lay.frame_meta[3 * f], R = lay.frame_meta[3 * f + 1], C = lay.frame_meta[3 * f + 2];
  const int32_t tiles_c = (C + kWideCols - 1) / kWideCols;
  const int32_t tr = t / tiles_c;
  const int32_t r0 = tr * kWideRows, c0 = (t - tr * tiles_c) * kWideCols;
  if (r0 >= R) return;  // (also covers t beyond this frame's tiles)
  const uint16_t* kframe = a.k + (size_t(unit) * lay.total_tokens + off) * kHeadDim;
  const int n = lane & 15, q = lane >> 4;

  // Output keys (row r0 + o, column c0 + n), clamped into the frame; the
  // clamped copies are never stored.
  bf16x8_t ha[kWideRows][4];
  float rnA[kWideRows];
#pragma unroll
  for (int o = 0; o < kWideRows; ++o)
    rnA[o] = load_key_operand(kframe, min(r0 + o, R - 1), min(c0 + n, C - 1), C, q, ha[o]);

  // Accumulator element (i, n) of block nb pairs output column c0 + 4 q + i
  // with neighbour column c0 - KR + 16 nb + n: dc = 16 nb + n - KR - 4 q - i.
  uint32_t near = 0, self = 0;  // bit 4 nb + i
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t d = 16 * nb + n - 4 * q - i;  // dc + KR
      const int32_t cc = c0 - KR + 16 * nb + n;
      if (d >= 0 && d <= 2 * KR && cc >= 0 && cc < C) near |= 1u << (4 * nb + i);
      if (d == KR) self |= 1u << (4 * nb + i);
    }

  float psum[kWideRows][4];
#pragma unroll
  for (int o = 0; o < kWideRows; ++o)
#pragma unroll
    for (int i = 0; i < 4; ++i) psum[o][i] = 0.0f;

  const uint32_t off_self = near & ~self;
  const int32_t rr0 = max(r0 - KR, 0), rr1 = min(r0 + kWideRows - 1 + KR, R - 1);
  // Neighbour row rr's B fragments: strip keys c0 - KR + 16 nb + n (clamped).
  auto fetch = [&](int32_t rr, uint4 (&v)[2][4]) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const uint16_t* src =
          kframe + (size_t(rr) * C + min(max(c0 - KR + 16 * nb + n, 0), C - 1)) * kHeadDim + q * 8;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) v[nb][kk] = *reinterpret_cast<const uint4*>(src + kk * 32);
    }
  };
  // One neighbour row; the next row's loads are issued first and stay in
  // flight under this row's matrix work.
  auto row = [&](int32_t rr, const uint4 (&v)[2][4], uint4 (&next)[2][4]) {
    if (rr < rr1) fetch(rr + 1, next);
    bf16x8_t hb[2][4];
    float sc_near[2][4], sc_off[2][4];  // the neighbour's inverse norm where the product counts, else 0
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float ss = 0.0f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        ss += sumsq8(v[nb][kk]);
        hb[nb][kk] = __builtin_bit_cast(bf16x8_t, v[nb][kk]);
      }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      const float rn = inv_norm(ss);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sc_near[nb][i] = (near >> (4 * nb + i)) & 1u ? rn : 0.0f;
        sc_off[nb][i] = (off_self >> (4 * nb + i)) & 1u ? rn : 0.0f;
      }
    }
#pragma unroll
    for (int o = 0; o < kWideRows; ++o) {
      const int32_t ro = r0 + o;
      if (ro >= R || rr < ro - KR || rr > ro + KR) continue;  // wave-uniform
      f32x4_t acc[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[o][kk], hb[nb][kk], acc[nb], 0, 0, 0);
      }
      if (rr == ro) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) psum[o][i] = fmaf(acc[nb][i], sc_off[nb][i], psum[o][i]);
      } else {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) psum[o][i] = fmaf(acc[nb][i], sc_near[nb][i], psum[o][i]);
      }
    }
  };
  uint4 bufA[2][4], bufB[2][4];
  fetch(rr0, bufA);
  for (int32_t rr = rr0; rr <= rr1; rr += 2) {
    row(rr, bufA, bufB);
    if (rr + 1 <= rr1) row(rr + 1, bufB, bufA);
  }

  float* phi = a.phi + size_t(unit) * lay.total_tokens + off;
#pragma unroll
  for (int o = 0; o < kWideRows; ++o)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float h = psum[o][i];
#pragma unroll
      for (int m = 1; m < 16; m <<= 1) h += __shfl_xor(h, m);
      const float rn_out = __shfl(rnA[o], 4 * q + i);  // inverse norm of output column c0 + 4 q + i
      const int32_t r = r0 + o, c = c0 + 4 * q + i;
      if (n == 0 && r < R && c < C) {
        const int32_t rows_in = min(r + KR, R - 1) - max(r - KR, 0) + 1;
        const int32_t cols_in = min(c + KR, C - 1) - max(c - KR, 0) + 1;
        const int32_t nn = rows_in * cols_in - 1;
        phi[size_t(r) * C + c] = nn > 0 ? 1.0f - h * rn_out / float(nn) : 0.0f;
      }
    }
}

// Phi = 0 on text tokens: work-group (g, unit) writes text run g (token_run),
// all runs at once.
__global__ __launch_bounds__(256) void css_text_kernel(CssArgs a) {
  const Layout& lay = a.lay;
  float* out = a.phi + size_t(blockIdx.y) * lay.total_tokens;
  int32_t b, e;
  token_run(lay, int32_t(blockIdx.x), false, &b, &e);
  for (int32_t j = b + int32_t(threadIdx.x); j < e; j += blockDim.x) out[j] = 0.0f;
}

}  // namespace

hipError_t launch_css_wide(const CssArgs& a, int32_t nbhd, hipStream_t stream) {
  hipLaunchKernelGGL(css_text_kernel, dim3(a.lay.n_frames + a.lay.n_seqs, a.lay.n_units), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.lay.n_frames == 0) return e;
  const int64_t logical = int64_t(a.lay.n_frames) * a.strips;  // a.strips: max over frames of 4 x 16 tiles
  const int64_t grid_x = ((logical + 3) / 4 + 7) / 8 * 8;
  const dim3 grid(unsigned(grid_x), a.lay.n_units);
  switch (nbhd) {
    case 5: hipLaunchKernelGGL(css_wide_kernel<2>, grid, dim3(256), 0, stream, a); break;
    case 7: hipLaunchKernelGGL(css_wide_kernel<3>, grid, dim3(256), 0, stream, a); break;
    case 9: hipLaunchKernelGGL(css_wide_kernel<4>, grid, dim3(256), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_css(const CssArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(css_text_kernel, dim3(a.lay.n_frames + a.lay.n_seqs, a.lay.n_units), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.lay.n_frames == 0) return e;
  const int64_t logical = int64_t(a.lay.n_frames) * a.strips;  // a.strips: max over frames of ceil(C / 14)
  const int64_t grid_x = (logical + 7) / 8 * 8;
  if (a.gate)
    hipLaunchKernelGGL(css_kernel<true>, dim3(unsigned(grid_x), a.lay.n_units), dim3(64), 0, stream, a);
  else
    hipLaunchKernelGGL(css_kernel<false>, dim3(unsigned(grid_x), a.lay.n_units), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
