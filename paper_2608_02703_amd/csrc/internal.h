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
  // persistent-grid sizes found with the occupancy API, keyed by kernel
  // variant; 0 = not computed yet
  std::atomic<int> grid_cache[64];
  // caller-owned hipEvent_t pair recorded around the head-streaming kernel
  std::atomic<void*> ev_start;
  std::atomic<void*> ev_stop;
};

namespace archead {

constexpr int64_t kDefaultGemvMaxM = 15;  // largest M on the decode kernel (measured crossover)
constexpr int kInt4Bias = 136;            // bf16 value of a nibble u is 128+u = 136+c

archead_status fail(archead_status s, const char* fmt, ...);
void clear_error();

// chunk = 32 consecutive INT4 codes = 16 bytes; lanes per row of the GEMV
int lanes_per_row(int64_t d);

// Workspace carve-up (byte offsets, each 256-aligned).
struct WsLayout {
  size_t t_off = 0;      // fp32 [M, r_c + r_r] (decode path)
  // many-token (MFMA) path only:
  size_t ts_off = 0;     // bf16 [M][blocks][4][16] t split into hi, mid, lo (and 0)
  size_t gb_off = 0;     // fp32 [n_mt][slots][256] slot biases
  size_t rat_off = 0;    // fp32 [n_vt][slots][256] scale ratios
  size_t fin_off = 0;    // fp32 [n_vt][256] final scales
  size_t wbf_off = 0;    // bf16 [r_c + r_r][d] factor codes of V_c and B_w
  size_t uc_off = 0;     // int8 [V][blocks][2][16] codes of U_c and A_w, padded, twice
  size_t part_off = 0;   // float2 [M, n_part] (CE)
  size_t tgt_off = 0;    // fp32 [M] (CE)
  size_t total = 0;
  int64_t n_part = 0;
};
WsLayout ws_layout(const archead_handle* h, int64_t M, archead_op op);
bool use_gemv(const archead_handle* h, int64_t M);

// grid of the GEMV kernel: persistent workgroups, at most one per 8 rows
int64_t gemv_grid(const archead_handle* h, int tok, bool ce);

}  // namespace archead
