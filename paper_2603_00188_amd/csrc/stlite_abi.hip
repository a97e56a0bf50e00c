// Host layer of libstlite: argument validation, workspace sizing, launch
// configuration and status codes for the C ABI declared in include/stlite.h.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>

#include "stlite.h"
#include "stlite_internal.h"

using namespace stlite;

namespace {

thread_local char g_last_error[512] = "";

stlite_status fail(stlite_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

stlite_status ok() {
  g_last_error[0] = '\0';
  return STLITE_OK;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// Host-side facts derived from the validated mirrors.
struct Facts {
  int64_t units;
  int64_t max_seq;
  int64_t total_hist_blocks;
  int64_t max_cur;
  int32_t rows, rows_pad, blocks, waves, row_blocks, balanced, chunk;
  int64_t total_chunks;
  int32_t sel_parts;    // parts per segment of the gate and top-B selections
  int32_t max_seq_frames;
};

Facts derive(const stlite_problem* p) {
  Facts f{};
  f.units = int64_t(p->n_layers) * p->n_kv_heads;
  const int32_t G = p->n_q_heads / p->n_kv_heads;
  f.rows = G * p->window;
  const int nb = (f.rows + 31) / 32;
  // ceil(nb / 2) waves (1..8), each holding at most two resident 32-row
  // blocks: at most one padded block.
  f.blocks = nb;
  f.row_blocks = nb >= 2 ? 2 : 1;
  f.waves = (nb + f.row_blocks - 1) / f.row_blocks;
  // 14 blocks (e.g. G = 7 query heads per KV head, window 64) run on 8 waves
  // instead of 7, two of the blocks split by key block between two waves, so
  // that each of the four SIMDs of a CU carries the same vector work.
  f.balanced = nb == 14 ? 1 : 0;
  if (f.balanced) f.waves = 8;
  f.rows_pad = f.waves * f.row_blocks * 32;
  // Key chunk per work-group of the score passes.  Their window queries fill
  // the register file (two waves per SIMD), so a CU holds 8 / waves of their
  // work-groups and the grid drains in rounds of 256 x that many work-groups
  // of (nearly) equal length: a last round with a few work-groups leaves the
  // chip idle for a whole chunk.  The chunk (a multiple of 64 keys between
  // 1024 and 16384; below 1024 keys the load of the group's window queries
  // outweighs the keys) minimises rounds x (tiles per chunk + ~4 tiles of
  // query load); with many sequences it is sized for >= 2048 work-groups.
  const int64_t work = f.units * p->total_tokens;
  if (p->n_seqs <= 256 && f.units > 0) {
    const int64_t slots = 256 * std::max(1, 8 / f.waves);
    int64_t best = -1, best_cost = 0;
    for (int64_t ch = 1024; ch <= 16384; ch += 64) {
      int64_t n = 0;
      for (int s = 0; s < p->n_seqs; ++s) n += ceil_div(p->h_cu_seqlens[s + 1] - p->h_cu_seqlens[s], ch);
      const int64_t cost = ceil_div(n * f.units, slots) * (ch / 64 + 4);
      if (best < 0 || cost < best_cost) {
        best = ch;
        best_cost = cost;
      }
    }
    f.chunk = int32_t(best);
  } else {
    int64_t ch = ceil_div(work, 2048);
    ch = ceil_div(ch, 64) * 64;
    f.chunk = int32_t(std::min<int64_t>(4096, std::max<int64_t>(1024, ch)));
  }
  for (int s = 0; s < p->n_seqs; ++s) {
    const int64_t L = p->h_cu_seqlens[s + 1] - p->h_cu_seqlens[s];
    f.max_seq = std::max(f.max_seq, L);
    f.total_chunks += ceil_div(L, f.chunk);
    const int32_t f0 = p->h_cu_frames[s], f1 = p->h_cu_frames[s + 1];
    f.max_seq_frames = std::max(f.max_seq_frames, f1 - f0);
    int64_t hist = 0;
    for (int32_t fi = f0; fi < f1; ++fi) {
      const int64_t n = int64_t(p->h_frame_meta[3 * fi + 1]) * p->h_frame_meta[3 * fi + 2];
      if (fi + 1 < f1)
        hist += n;
      else
        f.max_cur = std::max(f.max_cur, n);
    }
    f.total_hist_blocks += ceil_div(hist, kRhoRows);
  }
  // Selection parts: aim for >= 512 work-groups over all segments and for
  // parts of at most ~32768 tokens (the longest segment's part bounds the
  // pass), with parts of at least ~4096 tokens, at most 16.
  const int64_t segs = std::max<int64_t>(f.units * p->n_seqs, 1);
  int64_t parts = std::max(ceil_div(512, segs), ceil_div(f.max_seq, 32768));
  parts = std::min(parts, std::max<int64_t>(ceil_div(f.max_seq, 4096), 1));
  f.sel_parts = int32_t(std::min<int64_t>(std::max<int64_t>(parts, 1), 16));
  return f;
}

// Workspace of the four passes of one selection (gate or top-B): a row of
// 32-bit keys per unit (every sequence's keys starting 16-byte aligned), the
// part histograms of the three radix levels, the parts' counts below the
// level-1 prefix and the per-segment state.
size_t four_pass_bytes(const stlite_problem* p, const Facts& f) {
  const size_t segparts = size_t(f.units) * p->n_seqs * f.sel_parts;
  return align_up(size_t(f.units) * size_t(sel_key_stride(p->total_tokens, p->n_seqs)) * sizeof(uint32_t)) +
         2 * align_up(segparts * (2048 + 64) * sizeof(uint32_t)) + align_up(segparts * (1024 + 32) * sizeof(uint32_t)) +
         align_up(segparts * sizeof(int32_t)) + align_up(size_t(f.units) * p->n_seqs * 8 * sizeof(int32_t));
}

// Workspace of the splitter path: a code byte per token, the tile records,
// the candidate lists and the per-segment state.
size_t split_bytes(const stlite_problem* p, const Facts& f) {
  const size_t U = size_t(f.units);
  return align_up(U * size_t(sp_tile_stride(p->total_tokens, p->n_seqs)) * 256) +
         align_up(U * size_t(sp_tile_stride(p->total_tokens, p->n_seqs)) * 8 * sizeof(int32_t)) +
         align_up(U * size_t(sp_cand_stride(p->total_tokens, p->n_seqs)) * sizeof(uint2)) +
         align_up(U * p->n_seqs * kSpWords * sizeof(int32_t));
}

// Either path may run a call's selection (the diagnostic override below
// picks among them), so the workspace holds the larger of the two; they
// share its bytes.
size_t seg_bytes(const stlite_problem* p, const Facts& f) { return std::max(four_pass_bytes(p, f), split_bytes(p, f)); }

// Work-groups per segment of the splitter path's classify and emit passes:
// 32 tiles each (eight per wave) for the longest segment, fewer parts when
// that would exceed ~16k work-groups.
int32_t split_parts(const stlite_problem* p, const Facts& f) {
  const int64_t segs = std::max<int64_t>(f.units * p->n_seqs, 1);
  const int64_t tiles = std::max<int64_t>(ceil_div(f.max_seq, 256), 1);
  int64_t parts = ceil_div(tiles, 32);
  parts = std::min(parts, std::max<int64_t>(ceil_div(16384, segs), 1));
  return int32_t(std::max<int64_t>(parts, 1));
}

// The selection path.  By default segments of at most kSelResidentCapacity
// tokens run resident and longer ones take the splitter path.  The
// environment variable STLITE_SELECT_PATH overrides this for diagnostics and
// cross-checks: "four_pass", "split", "split_exact" (the splitter path with
// every segment resolved by its exact fallback) or "resident" (honoured when
// every segment fits).
void sel_path(const Facts& f, SelPlan& s) {
  const bool resident_ok = s.lds_frames && f.max_seq <= kSelResidentCapacity;
  s.path = resident_ok ? kSelPathResident : kSelPathSplit;
  s.split_exact = 0;
  const char* e = getenv("STLITE_SELECT_PATH");
  if (!e) return;
  if (!strcmp(e, "four_pass")) {
    s.path = kSelPathFourPass;
  } else if (!strcmp(e, "split")) {
    s.path = kSelPathSplit;
  } else if (!strcmp(e, "split_exact")) {
    s.path = kSelPathSplit;
    s.split_exact = 1;
  } else if (!strcmp(e, "resident") && resident_ok) {
    s.path = kSelPathResident;
  }
}

SelPlan sel_carve(const stlite_problem* p, const Facts& f, char* w) {
  const size_t segparts = size_t(f.units) * p->n_seqs * f.sel_parts;
  SelPlan s;
  s.parts = f.sel_parts;
  s.lds_frames = f.max_seq_frames <= kSelFrames ? 1 : 0;
  sel_path(f, s);
  s.split_parts = split_parts(p, f);
  s.split_tiles = int32_t(std::max<int64_t>(ceil_div(f.max_seq, 256), 1));
  {  // the splitter path's arrays, over the same bytes as the four passes' ones
    const size_t U = size_t(f.units);
    char* x = w;
    s.codes = reinterpret_cast<uint8_t*>(x);
    x += align_up(U * size_t(sp_tile_stride(p->total_tokens, p->n_seqs)) * 256);
    s.tiles = reinterpret_cast<int32_t*>(x);
    x += align_up(U * size_t(sp_tile_stride(p->total_tokens, p->n_seqs)) * 8 * sizeof(int32_t));
    s.cands = reinterpret_cast<uint2*>(x);
    x += align_up(U * size_t(sp_cand_stride(p->total_tokens, p->n_seqs)) * sizeof(uint2));
    s.sstate = reinterpret_cast<int32_t*>(x);
  }
  s.keys = reinterpret_cast<uint32_t*>(w);
  w += align_up(size_t(f.units) * size_t(sel_key_stride(p->total_tokens, p->n_seqs)) * sizeof(uint32_t));
  s.hist0 = reinterpret_cast<uint32_t*>(w);
  w += align_up(segparts * (2048 + 64) * sizeof(uint32_t));
  s.hist1 = reinterpret_cast<uint32_t*>(w);
  w += align_up(segparts * (2048 + 64) * sizeof(uint32_t));
  s.hist2 = reinterpret_cast<uint32_t*>(w);
  w += align_up(segparts * (1024 + 32) * sizeof(uint32_t));
  s.below = reinterpret_cast<int32_t*>(w);
  w += align_up(segparts * sizeof(int32_t));
  s.state = reinterpret_cast<int32_t*>(w);
  return s;
}

// TSG plan: historical-token table and rho block table.
size_t plan_bytes(const stlite_problem* p, const Facts& f) {
  return align_up(size_t(p->total_tokens) * sizeof(int32_t)) +
         align_up(size_t(std::max<int64_t>(f.total_hist_blocks, 1)) * sizeof(HistBlock));
}

// Carves the plan at w and, when `select` is set, the gate's selection keys after it.
void gate_carve(const stlite_problem* p, const Facts& f, char* w, bool select, GateArgs& g) {
  g.hist_tok = reinterpret_cast<int32_t*>(w);
  w += align_up(size_t(p->total_tokens) * sizeof(int32_t));
  g.blocks = reinterpret_cast<HistBlock*>(w);
  w += align_up(size_t(std::max<int64_t>(f.total_hist_blocks, 1)) * sizeof(HistBlock));
  g.sel = select ? sel_carve(p, f, w) : SelPlan{};
  g.tau = nullptr;
}

RhoArgs rho_args(const stlite_problem* p, const Facts& f, const uint16_t* k, float* rho, float* rn_cur,
                 const GateArgs& g) {
  RhoArgs r;
  r.lay = g.lay;
  r.sim = kSimCosine;
  r.k = k;
  r.rn_cur = rn_cur;
  r.rho = rho;
  r.hist_tok = g.hist_tok;
  r.blocks = g.blocks;
  r.total_hist_blocks = int32_t(f.total_hist_blocks);
  r.max_cur = int32_t(f.max_cur);
  return r;
}

Layout make_layout(const stlite_problem* p) {
  Layout l;
  l.cu_seqlens = p->cu_seqlens;
  l.cu_frames = p->cu_frames;
  l.frame_meta = p->frame_meta;
  l.cu_budget = p->cu_budget;
  l.n_seqs = p->n_seqs;
  l.n_frames = p->n_frames;
  l.n_units = p->n_layers * p->n_kv_heads;
  l.n_kv_heads = p->n_kv_heads;
  l.total_tokens = p->total_tokens;
  l.total_budget = p->total_budget;
  return l;
}

stlite_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(STLITE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

stlite_status check_ws(const stlite_problem* p, stlite_call call, const void* ws, size_t bytes) {
  size_t need = 0;
  stlite_status st = stlite_workspace_size(p, call, &need);
  if (st != STLITE_OK) return st;
  if (need > 0 && ws == nullptr) return fail(STLITE_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (bytes < need) return fail(STLITE_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0) return fail(STLITE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return STLITE_OK;
}

bool aligned16(const void* ptr) { return reinterpret_cast<uintptr_t>(ptr) % 16 == 0; }

// Decode attention: rows per work-group (aim for >= 2048 work-groups) and the
// chunk count over all sequences of a cache.
struct DecodePlan {
  const int32_t* h_cu_rows;
  int64_t total_rows;
  int32_t chunk;
  int64_t total_chunks;
};

DecodePlan decode_plan(const stlite_problem* p, bool compact) {
  DecodePlan d;
  d.h_cu_rows = compact ? p->h_cu_budget : p->h_cu_seqlens;
  d.total_rows = compact ? p->total_budget : p->total_tokens;
  const int64_t units = int64_t(p->n_layers) * p->n_kv_heads;
  int64_t ch = ceil_div(std::max<int64_t>(units * d.total_rows, 1), 2048);
  ch = ceil_div(ch, 64) * 64;
  d.chunk = int32_t(std::min<int64_t>(4096, std::max<int64_t>(256, ch)));
  d.total_chunks = 0;
  for (int s = 0; s < p->n_seqs; ++s) d.total_chunks += ceil_div(d.h_cu_rows[s + 1] - d.h_cu_rows[s], d.chunk);
  return d;
}

size_t decode_bytes(const stlite_problem* p, const DecodePlan& d) {
  const size_t parts = size_t(p->n_layers) * p->n_kv_heads * size_t(d.total_chunks) * 16;
  return 2 * align_up(parts * sizeof(float)) + align_up(parts * kHeadDim * sizeof(float));
}

}  // namespace

namespace stlite {

// Sets the calling thread's stlite_last_error() message for another source
// file of the library and returns st.
stlite_status report_error(stlite_status st, const char* msg) { return fail(st, "%s", msg); }

}  // namespace stlite

extern "C" {

int32_t stlite_abi_version(void) { return STLITE_ABI_VERSION; }

const char* stlite_status_string(stlite_status s) {
  switch (s) {
    case STLITE_OK: return "STLITE_OK";
    case STLITE_ERR_INVALID_ARG: return "STLITE_ERR_INVALID_ARG";
    case STLITE_ERR_UNSUPPORTED: return "STLITE_ERR_UNSUPPORTED";
    case STLITE_ERR_WORKSPACE: return "STLITE_ERR_WORKSPACE";
    case STLITE_ERR_HIP: return "STLITE_ERR_HIP";
  }
  return "STLITE_ERR_UNKNOWN";
}

const char* stlite_last_error(void) { return g_last_error; }

int64_t stlite_budget(int64_t L, int64_t beta_num, int64_t beta_den) {
  if (L < 0 || beta_num <= 0 || beta_den <= 0 || beta_num > beta_den) return -1;
  const __int128 prod = static_cast<__int128>(L) * beta_num;
  return static_cast<int64_t>(prod / beta_den);
}

constexpr int64_t kMaxFramePatches = int64_t(1) << 22;  // rows * cols of one frame

stlite_status stlite_validate(const stlite_problem* p) {
  if (!p) return fail(STLITE_ERR_INVALID_ARG, "problem is NULL");
  if (p->reserved != 0) return fail(STLITE_ERR_INVALID_ARG, "reserved field must be 0");
  if (p->n_layers < 1 || p->n_q_heads < 1 || p->n_kv_heads < 1)
    return fail(STLITE_ERR_INVALID_ARG, "n_layers, n_q_heads and n_kv_heads must be >= 1");
  if (p->n_q_heads % p->n_kv_heads != 0)
    return fail(STLITE_ERR_INVALID_ARG, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)",
                p->n_q_heads, p->n_kv_heads);
  if (p->head_dim != kHeadDim)
    return fail(STLITE_ERR_UNSUPPORTED, "head_dim %d: only %d is implemented", p->head_dim, kHeadDim);
  if (p->n_seqs < 1) return fail(STLITE_ERR_INVALID_ARG, "n_seqs must be >= 1");
  if (p->n_seqs > 65535) return fail(STLITE_ERR_UNSUPPORTED, "n_seqs %d: at most 65535 sequences", p->n_seqs);
  if (p->n_frames < 0) return fail(STLITE_ERR_INVALID_ARG, "n_frames must be >= 0");
  if (p->window < 1) return fail(STLITE_ERR_INVALID_ARG, "window must be >= 1");
  const int64_t G = p->n_q_heads / p->n_kv_heads;
  if (G * p->window > kMaxWindowRows)
    return fail(STLITE_ERR_UNSUPPORTED, "G * window = %lld exceeds %d", (long long)(G * p->window),
                kMaxWindowRows);
  if (!p->h_cu_seqlens || !p->h_cu_frames || !p->h_cu_budget || (p->n_frames > 0 && !p->h_frame_meta))
    return fail(STLITE_ERR_INVALID_ARG, "a host layout mirror is NULL");
  if (!p->cu_seqlens || !p->cu_frames || !p->cu_budget || (p->n_frames > 0 && !p->frame_meta))
    return fail(STLITE_ERR_INVALID_ARG, "a device layout array is NULL");
  if (p->h_cu_seqlens[0] != 0) return fail(STLITE_ERR_INVALID_ARG, "cu_seqlens[0] must be 0");
  if (p->h_cu_frames[0] != 0) return fail(STLITE_ERR_INVALID_ARG, "cu_frames[0] must be 0");
  if (p->h_cu_budget[0] != 0) return fail(STLITE_ERR_INVALID_ARG, "cu_budget[0] must be 0");
  for (int s = 0; s < p->n_seqs; ++s) {
    const int64_t a = p->h_cu_seqlens[s], b = p->h_cu_seqlens[s + 1];
    if (b - a > (int64_t(1) << 28))
      return fail(STLITE_ERR_UNSUPPORTED, "sequence %d has %lld tokens; at most 2^28 are supported", s, (long long)(b - a));
    if (b - a < p->window)
      return fail(STLITE_ERR_INVALID_ARG, "sequence %d has %lld tokens, fewer than the window %d", s,
                  (long long)(b - a), p->window);
    const int64_t B = int64_t(p->h_cu_budget[s + 1]) - p->h_cu_budget[s];
    if (B < 0 || B > b - a)
      return fail(STLITE_ERR_INVALID_ARG, "sequence %d: budget %lld outside [0, %lld]", s, (long long)B,
                  (long long)(b - a));
    const int32_t f0 = p->h_cu_frames[s], f1 = p->h_cu_frames[s + 1];
    if (f1 < f0 || f1 > p->n_frames)
      return fail(STLITE_ERR_INVALID_ARG, "cu_frames is not a prefix sum ending at n_frames");
    int64_t prev_end = a;
    for (int32_t f = f0; f < f1; ++f) {
      const int64_t off = p->h_frame_meta[3 * f], r = p->h_frame_meta[3 * f + 1], c = p->h_frame_meta[3 * f + 2];
      if (r < 1 || c < 1) return fail(STLITE_ERR_INVALID_ARG, "frame %d has an empty grid (%lld x %lld)", f,
                                      (long long)r, (long long)c);
      // A frame's keys are addressed by buffer descriptors of 32-bit byte
      // counts (256 bytes per patch): 2^22 patches keep them below 2^30.
      if (r * c > kMaxFramePatches)
        return fail(STLITE_ERR_UNSUPPORTED, "frame %d has %lld patches; at most 2^22 are supported", f,
                    (long long)(r * c));
      if (off < prev_end || off + r * c > b)
        return fail(STLITE_ERR_INVALID_ARG,
                    "frame %d [%lld, %lld) overlaps its predecessor or leaves sequence %d [%lld, %lld)", f,
                    (long long)off, (long long)(off + r * c), s, (long long)a, (long long)b);
      prev_end = off + r * c;
    }
  }
  if (p->h_cu_frames[p->n_seqs] != p->n_frames)
    return fail(STLITE_ERR_INVALID_ARG, "cu_frames[n_seqs] = %d but n_frames = %d", p->h_cu_frames[p->n_seqs],
                p->n_frames);
  if (p->total_tokens != p->h_cu_seqlens[p->n_seqs])
    return fail(STLITE_ERR_INVALID_ARG, "total_tokens %lld != cu_seqlens[n_seqs] %d", (long long)p->total_tokens,
                p->h_cu_seqlens[p->n_seqs]);
  if (p->total_budget != p->h_cu_budget[p->n_seqs])
    return fail(STLITE_ERR_INVALID_ARG, "total_budget %lld != cu_budget[n_seqs] %d", (long long)p->total_budget,
                p->h_cu_budget[p->n_seqs]);
  if (int64_t(p->n_layers) * p->n_kv_heads > 65535)
    return fail(STLITE_ERR_UNSUPPORTED, "more than 65535 (layer, kv head) units");
  return ok();
}

stlite_status stlite_workspace_size(const stlite_problem* p, stlite_call call, size_t* bytes) {
  if (!bytes) return fail(STLITE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = 0;
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  const Facts f = derive(p);
  const size_t per_token = size_t(f.units) * size_t(p->total_tokens);
  switch (call) {
    case STLITE_CALL_SCORE_WINDOW:
      *bytes = align_up(size_t(f.units) * f.total_chunks * f.rows_pad * sizeof(float2)) +
               align_up(size_t(f.units) * p->n_seqs * f.rows_pad * sizeof(float)) +
               align_up(size_t(f.units) * f.total_chunks * sizeof(int32_t));
      break;
    case STLITE_CALL_TSG_GATE:
      // rho scratch, current-frame norms, plan, selection
      *bytes = 2 * align_up(per_token * sizeof(float)) + plan_bytes(p, f) + seg_bytes(p, f);
      break;
    case STLITE_CALL_TSG_RHO:
      // current-frame norms, plan
      *bytes = align_up(per_token * sizeof(float)) + plan_bytes(p, f);
      break;
    case STLITE_CALL_TSG_RHO_CONCAT:
      // current-frame norms per layer, plan
      *bytes = align_up(size_t(p->n_layers) * p->total_tokens * sizeof(float)) + plan_bytes(p, f);
      break;
    case STLITE_CALL_TSG_THRESHOLD:
      *bytes = plan_bytes(p, f) + seg_bytes(p, f);
      break;
    case STLITE_CALL_SELECT_TOPK:
      *bytes = seg_bytes(p, f);
      break;
    case STLITE_CALL_CSS_SALIENCY:
    case STLITE_CALL_COMPACT_KV:
      *bytes = 0;
      break;
    case STLITE_CALL_DECODE_FULL:
    case STLITE_CALL_DECODE_COMPACT:
      *bytes = decode_bytes(p, decode_plan(p, call == STLITE_CALL_DECODE_COMPACT));
      break;
    default:
      return fail(STLITE_ERR_INVALID_ARG, "unknown call %d", int(call));
  }
  return ok();
}

stlite_status stlite_score_window(const stlite_problem* p, const uint16_t* q_win, const uint16_t* k,
                                  float* a_base, void* ws, size_t ws_bytes, void* stream) {
  stlite_status st = check_ws(p, STLITE_CALL_SCORE_WINDOW, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  if (!q_win || !k || !a_base) return fail(STLITE_ERR_INVALID_ARG, "q_win, k and a_base must be non-NULL");
  if (!aligned16(q_win) || !aligned16(k)) return fail(STLITE_ERR_INVALID_ARG, "q_win and k must be 16-byte aligned");
  const Facts f = derive(p);
  ScoreArgs a;
  a.lay = make_layout(p);
  a.q = q_win;
  a.k = k;
  a.a_base = a_base;
  a.partial = static_cast<float2*>(ws);
  const size_t part_bytes = align_up(size_t(f.units) * f.total_chunks * f.rows_pad * sizeof(float2));
  a.lse2 = reinterpret_cast<float*>(static_cast<char*>(ws) + part_bytes);
  a.redo = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + part_bytes +
                                      align_up(size_t(f.units) * p->n_seqs * f.rows_pad * sizeof(float)));
  a.n_q_heads = p->n_q_heads;
  a.group = p->n_q_heads / p->n_kv_heads;
  a.window = p->window;
  a.rows = f.rows;
  a.rows_pad = f.rows_pad;
  a.blocks = f.blocks;
  a.waves = f.waves;
  a.row_blocks = f.row_blocks;
  a.balanced = f.balanced;
  a.chunk = f.chunk;
  a.total_chunks = int32_t(f.total_chunks);
  return hip_status(launch_score_window(a, static_cast<hipStream_t>(stream)), "score_window launch");
}

static stlite_status css_common(const stlite_problem* p, int32_t nbhd, const uint16_t* k, const uint8_t* gate,
                                float* phi, void* stream);

stlite_status stlite_css_saliency(const stlite_problem* p, const uint16_t* k, const uint8_t* gate, float* phi,
                                  void* stream) {
  return css_common(p, 3, k, gate, phi, stream);
}

stlite_status stlite_css_saliency_nbhd(const stlite_problem* p, int32_t nbhd, const uint16_t* k, float* phi,
                                       void* stream) {
  return css_common(p, nbhd, k, nullptr, phi, stream);
}

static stlite_status css_common(const stlite_problem* p, int32_t nbhd, const uint16_t* k, const uint8_t* gate,
                                float* phi, void* stream) {
  if (nbhd != 3 && nbhd != 5 && nbhd != 7 && nbhd != 9)
    return fail(STLITE_ERR_INVALID_ARG, "nbhd must be 3, 5, 7 or 9 (got %d)", int(nbhd));
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (!k || !phi) return fail(STLITE_ERR_INVALID_ARG, "k and phi must be non-NULL");
  if (!aligned16(k)) return fail(STLITE_ERR_INVALID_ARG, "k must be 16-byte aligned");
  CssArgs a;
  a.lay = make_layout(p);
  a.k = k;
  a.gate = gate;
  a.phi = phi;
  int32_t strips = 1;
  if (nbhd == 3) {
    for (int32_t fi = 0; fi < p->n_frames; ++fi)
      strips = std::max<int32_t>(strips, (p->h_frame_meta[3 * fi + 2] + 13) / 14);
    a.strips = strips;
    return hip_status(launch_css(a, static_cast<hipStream_t>(stream)), "css_saliency launch");
  }
  for (int32_t fi = 0; fi < p->n_frames; ++fi)  // 4 x 16 output tiles of the widest frame
    strips = std::max<int32_t>(strips, ((p->h_frame_meta[3 * fi + 1] + 3) / 4) * ((p->h_frame_meta[3 * fi + 2] + 15) / 16));
  a.strips = strips;
  return hip_status(launch_css_wide(a, nbhd, static_cast<hipStream_t>(stream)), "css_saliency launch");
}

stlite_status stlite_tsg_gate(const stlite_problem* p, const uint16_t* k, float* rho, float* tau,
                              uint8_t* gate, void* ws, size_t ws_bytes, void* stream) {
  stlite_status st = check_ws(p, STLITE_CALL_TSG_GATE, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  if (!k || !gate) return fail(STLITE_ERR_INVALID_ARG, "k and gate must be non-NULL");
  if (!aligned16(k)) return fail(STLITE_ERR_INVALID_ARG, "k must be 16-byte aligned");
  const Facts f = derive(p);
  const size_t slab = align_up(size_t(f.units) * p->total_tokens * sizeof(float));
  char* w = static_cast<char*>(ws);
  GateArgs g;
  g.lay = make_layout(p);
  g.rho = rho ? rho : reinterpret_cast<float*>(w);
  g.rho_zero_fill = rho;
  g.gate = gate;
  gate_carve(p, f, w + 2 * slab, true, g);
  g.tau = tau;
  const RhoArgs r = rho_args(p, f, k, const_cast<float*>(g.rho), reinterpret_cast<float*>(w + slab), g);
  return hip_status(launch_tsg_gate(r, g, static_cast<hipStream_t>(stream)), "tsg_gate launch");
}

stlite_status stlite_tsg_rho(const stlite_problem* p, const uint16_t* k, float* rho, void* ws, size_t ws_bytes,
                             void* stream) {
  return stlite_tsg_similarity(p, STLITE_SIM_COSINE, k, rho, ws, ws_bytes, stream);
}

stlite_status stlite_tsg_similarity(const stlite_problem* p, stlite_similarity sim, const uint16_t* k, float* rho,
                                    void* ws, size_t ws_bytes, void* stream) {
  if (sim != STLITE_SIM_COSINE && sim != STLITE_SIM_DOT && sim != STLITE_SIM_NEG_L2)
    return fail(STLITE_ERR_INVALID_ARG, "sim must be STLITE_SIM_COSINE, _DOT or _NEG_L2");
  stlite_status st = check_ws(p, STLITE_CALL_TSG_RHO, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  if (!k || !rho) return fail(STLITE_ERR_INVALID_ARG, "k and rho must be non-NULL");
  if (!aligned16(k)) return fail(STLITE_ERR_INVALID_ARG, "k must be 16-byte aligned");
  const Facts f = derive(p);
  const size_t slab = align_up(size_t(f.units) * p->total_tokens * sizeof(float));
  char* w = static_cast<char*>(ws);
  GateArgs g;
  g.lay = make_layout(p);
  g.rho = rho;
  g.rho_zero_fill = rho;
  g.gate = nullptr;
  gate_carve(p, f, w + slab, false, g);
  RhoArgs r = rho_args(p, f, k, rho, reinterpret_cast<float*>(w), g);
  r.sim = int32_t(sim);
  return hip_status(launch_tsg_rho(r, g, static_cast<hipStream_t>(stream)), "tsg_rho launch");
}

stlite_status stlite_tsg_fixed_gate(const stlite_problem* p, const float* rho, float tau, uint8_t* gate,
                                    void* stream) {
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (!rho || !gate) return fail(STLITE_ERR_INVALID_ARG, "rho and gate must be non-NULL");
  if (std::isnan(tau)) return fail(STLITE_ERR_INVALID_ARG, "tau must not be NaN");
  GateArgs g{};
  g.lay = make_layout(p);
  g.rho = rho;
  g.rho_zero_fill = nullptr;
  g.gate = gate;
  return hip_status(launch_tsg_fixed_gate(g, tau, static_cast<hipStream_t>(stream)), "tsg_fixed_gate launch");
}

stlite_status stlite_tsg_threshold(const stlite_problem* p, const float* rho, float* tau, uint8_t* gate,
                                   void* ws, size_t ws_bytes, void* stream) {
  stlite_status st = check_ws(p, STLITE_CALL_TSG_THRESHOLD, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  if (!rho || !gate) return fail(STLITE_ERR_INVALID_ARG, "rho and gate must be non-NULL");
  const Facts f = derive(p);
  GateArgs g;
  g.lay = make_layout(p);
  g.rho = rho;
  g.rho_zero_fill = nullptr;
  g.gate = gate;
  gate_carve(p, f, static_cast<char*>(ws), true, g);
  g.tau = tau;
  return hip_status(launch_tsg_threshold(g, static_cast<hipStream_t>(stream)), "tsg_threshold launch");
}

stlite_status stlite_select_topk(const stlite_problem* p, const float* a_base, const float* phi,
                                 const uint8_t* gate, float alpha, int32_t* kept, float* score, void* ws,
                                 size_t ws_bytes, void* stream) {
  stlite_status st = check_ws(p, STLITE_CALL_SELECT_TOPK, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  if (!a_base || (!kept && p->total_budget > 0))
    return fail(STLITE_ERR_INVALID_ARG, "a_base and kept must be non-NULL");
  if (!(alpha >= 0.0f) || !std::isfinite(alpha))
    return fail(STLITE_ERR_INVALID_ARG, "alpha must be finite and >= 0");
  SelectArgs a;
  a.lay = make_layout(p);
  a.a_base = a_base;
  a.phi = phi;
  a.gate = gate;
  a.alpha = alpha;
  a.kept = kept;
  a.score = score;
  a.sel = sel_carve(p, derive(p), static_cast<char*>(ws));
  return hip_status(launch_select(a, static_cast<hipStream_t>(stream)), "select_topk launch");
}

static stlite_status compact_common(const stlite_problem* p, const uint16_t* k, const uint16_t* v,
                                    const int32_t* kept, int32_t per_layer, uint16_t* k_out, uint16_t* v_out,
                                    void* stream);

stlite_status stlite_compact_kv(const stlite_problem* p, const uint16_t* k, const uint16_t* v,
                                const int32_t* kept, uint16_t* k_out, uint16_t* v_out, void* stream) {
  return compact_common(p, k, v, kept, 0, k_out, v_out, stream);
}

stlite_status stlite_compact_kv_layer(const stlite_problem* p, const uint16_t* k, const uint16_t* v,
                                      const int32_t* kept_layer, uint16_t* k_out, uint16_t* v_out, void* stream) {
  return compact_common(p, k, v, kept_layer, 1, k_out, v_out, stream);
}

stlite_status stlite_mean_attention(const stlite_problem* p, const float* a_base, int32_t width, float* a_mean,
                                   void* stream) {
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (width < 1 || width % 2 == 0 || width > 2 * kMeanMaxRadius + 1)
    return fail(STLITE_ERR_INVALID_ARG, "width must be odd, 1 <= width <= %d (got %d)", 2 * kMeanMaxRadius + 1,
                width);
  if (!a_base || !a_mean) return fail(STLITE_ERR_INVALID_ARG, "a_base and a_mean must be non-NULL");
  if (a_base == a_mean) return fail(STLITE_ERR_INVALID_ARG, "a_mean must not alias a_base");
  return hip_status(launch_mean_attention(a_base, a_mean, make_layout(p), width, static_cast<hipStream_t>(stream)),
                    "mean_attention launch");
}

stlite_status stlite_layer_mean(const stlite_problem* p, const float* a_base, float* a_layer, void* stream) {
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (!a_base || !a_layer) return fail(STLITE_ERR_INVALID_ARG, "a_base and a_layer must be non-NULL");
  return hip_status(launch_layer_mean(a_base, a_layer, make_layout(p), static_cast<hipStream_t>(stream)),
                    "layer_mean launch");
}

stlite_status stlite_tsg_rho_concat(const stlite_problem* p, const uint16_t* k, float* rho_layer, void* ws,
                                    size_t ws_bytes, void* stream) {
  stlite_status st = check_ws(p, STLITE_CALL_TSG_RHO_CONCAT, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  if (p->n_kv_heads != 2 && p->n_kv_heads != 4)
    return fail(STLITE_ERR_UNSUPPORTED, "the concatenated key space is implemented for 2 or 4 kv heads (got %d)",
                p->n_kv_heads);
  if (!k || !rho_layer) return fail(STLITE_ERR_INVALID_ARG, "k and rho_layer must be non-NULL");
  if (!aligned16(k)) return fail(STLITE_ERR_INVALID_ARG, "k must be 16-byte aligned");
  const Facts f = derive(p);
  char* w = static_cast<char*>(ws);
  GateArgs g{};
  g.lay = make_layout(p);
  g.lay.n_units = p->n_layers;  // per-layer output: rho_layer is zero-filled over [n_layers][L]
  g.lay.n_kv_heads = 1;
  g.rho = rho_layer;
  g.rho_zero_fill = rho_layer;
  g.gate = nullptr;
  const size_t slab = align_up(size_t(p->n_layers) * p->total_tokens * sizeof(float));
  gate_carve(p, f, w + slab, false, g);
  RhoArgs r = rho_args(p, f, k, rho_layer, reinterpret_cast<float*>(w), g);
  r.lay = make_layout(p);
  return hip_status(launch_tsg_rho_concat(r, g, static_cast<hipStream_t>(stream)), "tsg_rho_concat launch");
}

stlite_status stlite_css_saliency_concat(const stlite_problem* p, const uint16_t* k, float* phi_layer, void* stream) {
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (p->n_kv_heads != 2 && p->n_kv_heads != 4)
    return fail(STLITE_ERR_UNSUPPORTED, "the concatenated key space is implemented for 2 or 4 kv heads (got %d)",
                p->n_kv_heads);
  if (!k || !phi_layer) return fail(STLITE_ERR_INVALID_ARG, "k and phi_layer must be non-NULL");
  if (!aligned16(k)) return fail(STLITE_ERR_INVALID_ARG, "k must be 16-byte aligned");
  CssArgs a;
  a.lay = make_layout(p);
  a.k = k;
  a.gate = nullptr;
  a.phi = phi_layer;
  int32_t strips = 1;
  const int32_t rows = p->n_kv_heads >= 4 ? 1 : 2;  // output rows per wave tile (css_cat_kernel)
  for (int32_t fi = 0; fi < p->n_frames; ++fi)      // wave tiles of the largest frame
    strips = std::max<int32_t>(strips, ((p->h_frame_meta[3 * fi + 1] + rows - 1) / rows) *
                                           ((p->h_frame_meta[3 * fi + 2] + 15) / 16));
  a.strips = strips;
  return hip_status(launch_css_concat(a, static_cast<hipStream_t>(stream)), "css_saliency_concat launch");
}

static stlite_status compact_common(const stlite_problem* p, const uint16_t* k, const uint16_t* v,
                                    const int32_t* kept, int32_t per_layer, uint16_t* k_out, uint16_t* v_out,
                                    void* stream) {
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (p->total_budget == 0) return ok();
  if (!k || !v || !kept || !k_out || !v_out)
    return fail(STLITE_ERR_INVALID_ARG, "k, v, kept, k_out and v_out must be non-NULL");
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out))
    return fail(STLITE_ERR_INVALID_ARG, "k, v, k_out and v_out must be 16-byte aligned");
  CompactArgs a;
  a.lay = make_layout(p);
  a.k = k;
  a.v = v;
  a.kept = kept;
  a.kept_per_layer = per_layer;
  a.k_out = k_out;
  a.v_out = v_out;
  return hip_status(launch_compact(a, static_cast<hipStream_t>(stream)), "compact_kv launch");
}

stlite_status stlite_kept_overlap(const stlite_problem* p, const int32_t* kept_a, const int32_t* kept_b,
                                  int32_t* hits, void* stream) {
  stlite_status st = stlite_validate(p);
  if (st != STLITE_OK) return st;
  if (!hits) return fail(STLITE_ERR_INVALID_ARG, "hits must be non-NULL");
  if (p->total_budget > 0 && (!kept_a || !kept_b))
    return fail(STLITE_ERR_INVALID_ARG, "kept_a and kept_b must be non-NULL");
  OverlapArgs a;
  a.lay = make_layout(p);
  a.kept_a = kept_a;
  a.kept_b = kept_b;
  a.hits = hits;
  int64_t spans = 1;
  for (int32_t s = 0; s < p->n_seqs; ++s)
    spans = std::max<int64_t>(spans, (int64_t(p->h_cu_seqlens[s + 1]) - p->h_cu_seqlens[s] + 65535) / 65536);
  a.spans_per_seq = int32_t(spans);
  return hip_status(launch_kept_overlap(a, static_cast<hipStream_t>(stream)), "kept_overlap launch");
}

stlite_status stlite_decode_attention(const stlite_problem* p, stlite_cache cache, const uint16_t* q_dec,
                                      const uint16_t* k, const uint16_t* v, float* out, void* ws,
                                      size_t ws_bytes, void* stream) {
  if (cache != STLITE_CACHE_FULL && cache != STLITE_CACHE_COMPACT)
    return fail(STLITE_ERR_INVALID_ARG, "cache must be STLITE_CACHE_FULL or STLITE_CACHE_COMPACT");
  const bool compact = cache == STLITE_CACHE_COMPACT;
  stlite_status st = check_ws(p, compact ? STLITE_CALL_DECODE_COMPACT : STLITE_CALL_DECODE_FULL, ws, ws_bytes);
  if (st != STLITE_OK) return st;
  const int32_t G = p->n_q_heads / p->n_kv_heads;
  if (G > 16) return fail(STLITE_ERR_UNSUPPORTED, "decode attention needs G <= 16 (G = %d)", G);
  const DecodePlan d = decode_plan(p, compact);
  if (!q_dec || !out || (d.total_rows > 0 && (!k || !v)))
    return fail(STLITE_ERR_INVALID_ARG, "q_dec, out, k and v must be non-NULL");
  if (!aligned16(q_dec) || !aligned16(k) || !aligned16(v))
    return fail(STLITE_ERR_INVALID_ARG, "q_dec, k and v must be 16-byte aligned");
  DecodeArgs a;
  a.lay = make_layout(p);
  a.q = q_dec;
  a.k = k;
  a.v = v;
  a.cu_rows = compact ? p->cu_budget : p->cu_seqlens;
  a.total_rows = d.total_rows;
  a.out = out;
  const size_t parts = size_t(a.lay.n_units) * size_t(d.total_chunks) * 16;
  a.pm = static_cast<float*>(ws);
  a.pl = reinterpret_cast<float*>(static_cast<char*>(ws) + align_up(parts * sizeof(float)));
  a.po = reinterpret_cast<float*>(static_cast<char*>(ws) + 2 * align_up(parts * sizeof(float)));
  a.n_q_heads = p->n_q_heads;
  a.group = G;
  a.chunk = d.chunk;
  a.total_chunks = int32_t(d.total_chunks);
  return hip_status(launch_decode(a, static_cast<hipStream_t>(stream)), "decode_attention launch");
}

}  // extern "C"
