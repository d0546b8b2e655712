// Host-side internals shared by the host translation unit and the HIP one.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <atomic>

#include "archead.h"

struct archead_handle {
  archead_desc desc;
  archead_ptrs ptrs;
  int device;             // HIP device the buffers live on
  int n_cu;               // compute units of that device
  std::atomic<int64_t> gemv_max_m;
  std::atomic<int64_t> dec_min_m;   // M range of the MFMA decode kernel
  std::atomic<int64_t> dec_max_m;   // (empty when max < min)
  std::atomic<int64_t> mid_min_m;   // M range of the several-token kernel
  std::atomic<int64_t> mid_max_m;
  // archead_set_launch values (0 = built-in; the spin limit -1 = built-in)
  std::atomic<int64_t> launch[ARCHEAD_LAUNCH_KNOBS];
  // persistent-grid sizes found with the occupancy API, keyed by kernel
  // variant; 0 = not computed yet
  std::atomic<int> grid_cache[128];
  // caller-owned hipEvent_t pair recorded around the head-streaming kernel
  std::atomic<void*> ev_start;
  std::atomic<void*> ev_stop;
  // caller-owned device buffer holding the many-token kernel's tables
  // derived from the head (archead_prepare), or null: built per call
  std::atomic<char*> prep;
};

namespace archead {

constexpr int64_t kDefaultGemvMaxM = 15;  // largest M on the decode kernel (measured crossover)
constexpr int64_t kDefaultDecMinM = 2;    // M range of the MFMA decode kernel (one
constexpr int64_t kDefaultDecMaxM = 32;   // token streams faster through the GEMV)
constexpr int64_t kDefaultMidMaxM = 32;   // largest M of the several-token kernel (one pass)
constexpr int kDefaultSpinLimit = 1 << 16;   // polls of the stage-1 exchange before the fallback
constexpr int kInt4Bias = 136;            // bf16 value of a nibble u is 128+u = 136+c
constexpr int kDecTok = 16;               // tokens per pass of the MFMA decode kernel
constexpr int kDecWaves = 8;              // waves per workgroup of the MFMA decode kernel
constexpr int64_t kLdsBytes = 160 * 1024; // LDS per workgroup on gfx950
constexpr int kMidTokMax = 32;            // tokens per tile of the several-token kernel
constexpr int kMidWindow = 256;           // elements of d per x window of that kernel
constexpr int kMidWaveCount = 8;          // its waves per workgroup
constexpr int kTopKMaxK = 64;             // largest k of archead_logits_topk (lanes of a wave)
constexpr int64_t kTopKChunk = 256;       // tokens per chunk of the unfused top-k
constexpr int kTopKMergeBlock = 1024;     // threads of the round-based top-k merge workgroup
constexpr int kTopKMergeC = 8;            // candidates per thread of that merge (else the scan merge)

archead_status fail(archead_status s, const char* fmt, ...);
void clear_error();

// Device address of the static workspace of archead_logits_noalloc on
// `device` (the current device), taken once per device; called by
// archead_create.
archead_status scratch_setup(int device);

// bytes per vocabulary row of core_u (int8 codes, or ARCHEAD_I5 words)
int64_t core_u_row_bytes(const archead_desc& d);
// how the kernels read the factor codes: 0 aligned int8 (ranks multiples of
// 4); 1 int8 of any rank; 2 with the core-left codes in ARCHEAD_I5 words
int gen_codes(const archead_desc& d);

// chunk = 32 consecutive INT4 codes = 16 bytes; lanes per row of the GEMV
int lanes_per_row(const archead_desc& d);

// Workspace carve-up (byte offsets, each 256-aligned).
// kernel family serving a call
enum class Path { kDec, kMid, kGemv, kTiled };

struct WsLayout {
  size_t tst_off = 0;    // u64 [M, r_c + r_r] stamped t (decode and several-token kernels)
  // many-token (MFMA) path only:
  size_t ts_off = 0;     // bf16 [M][blocks][4][16] t split into hi, mid, lo (and 0)
  size_t gb_off = 0;     // fp32 [n_mt][slots][256] slot biases
  size_t rat_off = 0;    // fp32 [n_vt][slots][256] scale ratios
  size_t fin_off = 0;    // fp32 [n_vt][256] final scales
  size_t wbf_off = 0;    // bf16 [r_c + r_r][d] factor codes of V_c and B_w
  size_t uc_off = 0;     // int8 [V][blocks][2][16] codes of U_c and A_w, padded, twice
  size_t s1p_off = 0;    // fp32 [ksplit][M][r_c + r_r] stage-1 partials (split along d)
  size_t part_off = 0;   // float2 [M, n_part] (CE)
  size_t tgt_off = 0;    // fp32 [M] (CE)
  size_t pidx_off = 0;   // int32 [M, n_part] (argmax)
  // top-k: fused (single token on the decode GEMV) or over chunks of up to
  // kTopKChunk tokens whose fp32 logits go to lg_off, computed with the
  // workspace at in_off
  bool tk_fused = false;
  int64_t tk_chunk = 0;   // tokens per chunk (unfused)
  size_t tk_lg_off = 0;   // fp32 [chunk][V]
  size_t tk_in_off = 0;   // workspace of the chunk's logits call
  size_t tk_pv_off = 0;   // fp32 [chunk or 1][n_part][kTopKMax] partial lists
  size_t tk_pi_off = 0;   // int32, the same shape
  Path tk_path = Path::kGemv;   // kernel of the chunks' logits (that of the whole M)
  // fidelity against a dense head: the tiled path's layout, then
  size_t fid_off = 0;     // [M][n_vt] per-tile statistics (32 bytes each)
  size_t bref_off = 0;    // fp32 [M] packed logit at the dense top-1
  size_t total = 0;
  int64_t n_part = 0;
};
WsLayout ws_layout(const archead_handle* h, int64_t M, archead_op op);
WsLayout ws_layout_path(const archead_handle* h, int64_t M, archead_op op, Path path);

// The many-token kernel's tables that depend on the head only (scale
// ratios, final scales, bf16 V_c / B_w codes, paired U_c / A_w codes):
// offsets from the start of their block, in the workspace or in a prepared
// buffer (the same layout in both).
struct PrepLayout {
  size_t rat_off = 0, fin_off = 0, wbf_off = 0, uc_off = 0, total = 0;
};
PrepLayout prep_layout(const archead_handle* h);
bool use_gemv(const archead_handle* h, int64_t M);

// MFMA decode kernel: its LDS layout for a pass of `tok` tokens, the most
// tokens per pass the LDS holds (0: the head shape is not supported), and
// whether a call with M tokens runs on it.
struct DecLds {
  int xstr = 0, tstr = 0, off_bias = 0, off_t = 0, off_red = 0, total = 0;
  int kcu = 0, kca = 0;   // expansion K-chunks of 32 rank dimensions (U_c, A_w)
};
DecLds dec_lds(const archead_desc& d, int tok);
int dec_tokens_per_pass(const archead_desc& d);
bool use_dec(const archead_handle* h, int64_t M);

// Several-token kernel: LDS layout for its tiles of kMidTokMax tokens, whether the
// head shape is supported, and whether a call with M tokens runs on it.
struct MidLds {
  int tstr = 0, off_bias = 0, off_red = 0, off_y = 0, off_idx = 0, off_sc = 0, total = 0;
  int kcu = 0, kca = 0;
};
MidLds mid_lds(const archead_desc& d);
bool mid_supported(const archead_desc& d);
bool use_mid(const archead_handle* h, int64_t M);

// Built-in M ranges for a head shape: {dec_min, dec_max, mid_min, mid_max}.
// Where the several-token kernel applies, the MFMA decode kernel keeps the M
// it serves in one pass and the several-token kernel takes over from there
// up to kDefaultMidMaxM (measured crossovers); otherwise the decode kernel
// keeps its first M .. kDefaultDecMaxM.  Its first M is kDefaultDecMinM.
void default_ranges(const archead_desc& d, int64_t (&r)[4]);

// The kernel a call with M tokens runs on: the MFMA decode kernel, the
// several-token kernel, the decode GEMV or the tiled MFMA kernel, in that
// order of preference where the M ranges and the head shape allow.
Path choose_path(const archead_handle* h, int64_t M);

// grid of the GEMV kernel: persistent workgroups, at most one per 8 rows
int64_t gemv_grid(const archead_handle* h, int tok, bool ce, bool topk = false);

struct DecGrid {
  int prod_blocks = 0;          // stage-1 producer workgroups (first in the grid)
  int64_t consumer_blocks = 0;  // workgroups streaming the head
  int64_t n_waves = 0;          // consumer waves with work
  int64_t n_units = 0;          // units of 16 vocabulary rows
};
DecGrid dec_grid(const archead_handle* h);

struct MidGrid {
  int prod_blocks = 0;          // stage-1 producer workgroups (first in the grid)
  int64_t cblocks = 0;          // consumer workgroups (balanced ranges of units)
  int64_t n_units = 0;
};
MidGrid mid_grid(const archead_handle* h);

}  // namespace archead
