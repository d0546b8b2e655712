// Host-only part of the ARCHead C ABI: descriptor checks, byte accounting,
// INT4 packing and error reporting.  No HIP calls, so it also builds with a
// plain C++ compiler for the CPU tests.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "internal.h"

namespace archead {

static thread_local char g_err[512];

archead_status fail(archead_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

void clear_error() { g_err[0] = 0; }

int64_t core_u_row_bytes(const archead_desc& d) {
  return d.core_u_dtype == ARCHEAD_I5 ? 4 * ((d.r_c + 5) / 6) : d.r_c;
}

int gen_codes(const archead_desc& d) {
  if (d.core_u_dtype == ARCHEAD_I5 && d.r_c) return 2;
  return d.r_c % 4 || d.r_r % 4 ? 1 : 0;
}

int lanes_per_row(const archead_desc& d) {
  // a segment of 16 lanes per row reads 256 contiguous bytes per row and 4
  // rows per load instruction, which streams faster than one row per
  // instruction; wider segments only where the rank-r codes of a row would
  // not fit as 2 dwords per lane otherwise
  const int64_t chunks = d.d / 32;
  int lpr = 16;
  while (lpr > 1 && chunks % lpr) lpr >>= 1;
  const int64_t r4 = (d.r_c + d.r_r) / 4;
  while (lpr < 64 && r4 > 2 * lpr && chunks % (2 * lpr) == 0) lpr *= 2;
  // and where a row's group scales would not fit one dword per segment lane
  // (2 fp16 scales or 4 8-bit codes per lane: g = 64 with fp16 scales at
  // d = 4096 takes 32 lanes); the general-code variants keep 8 or 16
  const int64_t gpl = d.scale_dtype == ARCHEAD_U8 ? 4 : 2;
  if (!gen_codes(d))
    while (lpr < 64 && d.d / d.g > gpl * lpr && chunks % (2 * lpr) == 0) lpr *= 2;
  return lpr;
}

bool use_gemv(const archead_handle* h, int64_t M) {
  // the many-token kernel stages 64 codes of one scale group at a time
  return M <= h->gemv_max_m.load(std::memory_order_relaxed) || h->desc.g % 64 != 0;
}

DecLds dec_lds(const archead_desc& d, int tok) {
  DecLds l;
  l.kcu = int((d.r_c + 31) / 32);
  l.kca = int((d.r_r + 31) / 32);
  l.xstr = int(2 * d.d + 16);                   // +16 bytes: rows start on different banks
  l.tstr = (l.kcu + l.kca) * 32 + 8;            // bf16 elements, +16 bytes likewise
  l.off_bias = tok * l.xstr;
  l.off_t = l.off_bias + int(d.d / d.g) * kDecTok * 4;
  l.off_red = l.off_t + 3 * tok * l.tstr * 2;   // t as three bf16 parts
  l.total = l.off_red + kDecWaves * kDecTok * (8 + 4);   // softmax and argmax partials
  return l;
}

int dec_tokens_per_pass(const archead_desc& d) {
  // group sizes of 1, 2 or 4 code words per lane, walked 4 groups at a time;
  // at most 64 groups per row (two scale loads per unit); factor code rows
  // read as dwords; at most 128 dimensions per factor (4 K-chunks)
  if (d.g != 32 && d.g != 64 && d.g != 128) return 0;
  // 8-bit scale codes: all 64 groups of a row in one 16-byte load per lane
  if ((d.d / d.g) % 4 || d.d / d.g > 64) return 0;
  if (d.r_c > 128 || d.r_r > 128) return 0;
  // byte offsets of the code buffer stay 32-bit
  if (d.V * (d.d / 2) >= (int64_t(1) << 31)) return 0;
  for (int tok = kDecTok; tok >= 1; --tok)
    if (dec_lds(d, tok).total <= kLdsBytes) return tok;
  return 0;
}

bool use_dec(const archead_handle* h, int64_t M) {
  return M >= h->dec_min_m.load(std::memory_order_relaxed) &&
         M <= h->dec_max_m.load(std::memory_order_relaxed) && dec_tokens_per_pass(h->desc) > 0;
}

MidLds mid_lds(const archead_desc& d) {
  MidLds l;
  const int tm = kMidTokMax;
  l.kcu = int((d.r_c + 31) / 32);
  l.kca = int((d.r_r + 31) / 32);
  l.tstr = (l.kcu + l.kca) * 32 + 8;            // bf16 elements, +16 bytes: rows on different banks
  const int xwin = 2 * tm * (2 * kMidWindow + 16);   // two x windows, 16 bytes of padding per row
  const int tbytes = 3 * tm * l.tstr * 2;       // t as three bf16 parts (over the windows)
  l.off_bias = xwin > tbytes ? xwin : tbytes;
  l.off_red = l.off_bias + 2 * int(kMidWindow / d.g) * tm * 4;
  l.off_y = l.off_red + kMidWaveCount * tm * 8;
  l.off_idx = l.off_y + tm * 8;                 // argmax partials [waves][tm]
  l.off_sc = l.off_idx + kMidWaveCount * tm * 4; // per wave: [units][16 rows][d/g + 2] fp16
  const int nu = 3;                             // units per wave and pass
  l.total = l.off_sc + kMidWaveCount * nu * 16 * int(2 * (d.d / d.g) + 4);
  return l;
}

bool mid_supported(const archead_desc& d) {
  // groups of 64 or 128 codes, walked two windows of 256 elements at a time,
  // at most 64 groups per row (a unit's scales staged in LDS), factor code rows
  // read as dwords, at most 128 dimensions per factor (4 K-chunks)
  if (d.g != 64 && d.g != 128) return false;
  if (d.d % (2 * kMidWindow) || d.d / d.g > 64) return false;
  if (d.r_c > 128 || d.r_r > 128) return false;
  return mid_lds(d).total <= kLdsBytes;
}

// Two tokens: the GEMV's cost grows about 1.3x from one token to two on
// every measured head, the MFMA decode kernel's not at all, and with its
// code loads on the default cache policy its cost at two tokens is at or
// below the GEMV's on every measured head (M = 2: Qwen shape 64.5 against
// 76.4 us; Gemma shape 75.4 against 86.8; 128k head, ranks 128 / 64, 126.0
// against 127.0), so two tokens take it everywhere it applies.
static int64_t dec_min_m(const archead_desc&) { return kDefaultDecMinM; }

void default_ranges(const archead_desc& d, int64_t (&r)[4]) {
  const int tpp = dec_tokens_per_pass(d);
  if (mid_supported(d) && tpp > 0) {
    r[0] = dec_min_m(d);
    r[1] = tpp;
    r[2] = tpp + 1;
    // at d >= 8192 the tiled kernel overtakes it from 24 tokens on (128k
    // head: 198 / 224 us at M = 24 / 32 against 201 / 202 tiled)
    r[3] = d.d >= 8192 ? 24 : kDefaultMidMaxM;
  } else {
    r[0] = dec_min_m(d);
    r[1] = kDefaultDecMaxM;
    r[2] = 1;
    r[3] = 0;
  }
}

bool use_mid(const archead_handle* h, int64_t M) {
  return M >= h->mid_min_m.load(std::memory_order_relaxed) &&
         M <= h->mid_max_m.load(std::memory_order_relaxed) && mid_supported(h->desc);
}

Path choose_path(const archead_handle* h, int64_t M) {
  if (use_dec(h, M)) return Path::kDec;
  if (use_mid(h, M)) return Path::kMid;
  if (use_gemv(h, M)) return Path::kGemv;
  return Path::kTiled;
}

}  // namespace archead

using namespace archead;

extern "C" {

const char* archead_status_str(archead_status s) {
  switch (s) {
    case ARCHEAD_OK: return "ok";
    case ARCHEAD_E_INVALID_ARG: return "invalid argument";
    case ARCHEAD_E_MISALIGNED: return "misaligned pointer or stride";
    case ARCHEAD_E_UNSUPPORTED: return "unsupported device or shape";
    case ARCHEAD_E_WORKSPACE: return "workspace too small";
    case ARCHEAD_E_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* archead_last_error(void) { return archead::g_err; }

archead_status archead_validate_desc(const archead_desc* p) {
  if (!p) return fail(ARCHEAD_E_INVALID_ARG, "desc is NULL");
  const archead_desc& d = *p;
  if (d.abi_version != ARCHEAD_ABI_VERSION)
    return fail(ARCHEAD_E_INVALID_ARG, "abi_version %u, library is %u",
                d.abi_version, ARCHEAD_ABI_VERSION);
  if (d.V <= 0 || d.d <= 0 || d.g <= 0)
    return fail(ARCHEAD_E_INVALID_ARG, "V, d and g must be positive");
  if (d.V > (int64_t(1) << 31) - 1 || d.d > 16384)
    return fail(ARCHEAD_E_UNSUPPORTED, "V must be < 2^31 and d <= 16384");
  if (d.g % 32) return fail(ARCHEAD_E_INVALID_ARG, "g = %lld is not a multiple of 32", (long long)d.g);
  if (d.d % d.g) return fail(ARCHEAD_E_INVALID_ARG, "g = %lld does not divide d = %lld", (long long)d.g, (long long)d.d);
  if (d.r_c < 0 || d.r_r < 0) return fail(ARCHEAD_E_INVALID_ARG, "ranks must be >= 0");
  if (d.r_c + d.r_r > 1024) return fail(ARCHEAD_E_UNSUPPORTED, "r_c + r_r must be <= 1024");
  const int64_t gs[2] = {d.g_v, d.g_b};
  const int64_t rk[2] = {d.r_c, d.r_r};
  for (int i = 0; i < 2; ++i) {
    if (rk[i] == 0) continue;
    if (gs[i] <= 0 || gs[i] % 32 || d.d % gs[i])
      return fail(ARCHEAD_E_INVALID_ARG, "%s = %lld must divide d and be a multiple of 32",
                  i ? "g_b" : "g_v", (long long)gs[i]);
  }
  if (d.int4_encoding != ARCHEAD_INT4_V1)
    return fail(ARCHEAD_E_INVALID_ARG, "unknown int4_encoding %d", d.int4_encoding);
  if (d.scale_dtype != ARCHEAD_F16 && d.scale_dtype != ARCHEAD_U8)
    return fail(ARCHEAD_E_UNSUPPORTED, "scale_dtype must be ARCHEAD_F16 or ARCHEAD_U8");
  if (d.factor_dtype != ARCHEAD_I8)
    return fail(ARCHEAD_E_UNSUPPORTED, "factor_dtype must be ARCHEAD_I8");
  if (d.core_u_dtype != ARCHEAD_I8 && d.core_u_dtype != ARCHEAD_I5)
    return fail(ARCHEAD_E_UNSUPPORTED, "core_u_dtype must be ARCHEAD_I8 or ARCHEAD_I5");
  return ARCHEAD_OK;
}

uint64_t archead_packed_bytes(const archead_desc* p) {
  if (archead_validate_desc(p) != ARCHEAD_OK) return 0;
  const archead_desc& d = *p;
  const uint64_t V = d.V, D = d.d;
  uint64_t b = V * D / 2;                                     // residual codes
  if (d.scale_dtype == ARCHEAD_U8)
    b += V * (D / d.g) + V * 2;                                // 8-bit group codes + fp16 row scales
  else
    b += V * (D / d.g) * 2;                                    // fp16 group scales
  if (d.r_c) b += V * uint64_t(core_u_row_bytes(d)) + V * 2 + d.r_c * D + d.r_c * (D / d.g_v) * 2;
  if (d.r_r) b += V * d.r_r + V * 2 + d.r_r * D + d.r_r * (D / d.g_b) * 2;
  return b;
}

archead_status archead_pack_int5(const int8_t* codes, int64_t rows, int64_t r, uint32_t* packed) {
  if (!codes || !packed || rows < 0 || r < 1)
    return fail(ARCHEAD_E_INVALID_ARG, "pack_int5: bad pointers or shape (r >= 1)");
  const int64_t w5 = (r + 5) / 6;
  for (int64_t row = 0; row < rows; ++row) {
    for (int64_t w = 0; w < w5; ++w) {
      uint32_t q = 0;
      for (int64_t j = 0; j < 6 && 6 * w + j < r; ++j) {
        const int v = codes[row * r + 6 * w + j];
        if (v < -16 || v > 15)
          return fail(ARCHEAD_E_INVALID_ARG, "pack_int5: code %d out of [-16, 15] at (%lld, %lld)",
                      v, (long long)row, (long long)(6 * w + j));
        q |= (uint32_t(v) & 31u) << (5 * j);
      }
      packed[row * w5 + w] = q;
    }
  }
  return ARCHEAD_OK;
}

archead_status archead_unpack_int5(const uint32_t* packed, int64_t rows, int64_t r,
                                   int8_t* codes) {
  if (!codes || !packed || rows < 0 || r < 1)
    return fail(ARCHEAD_E_INVALID_ARG, "unpack_int5: bad pointers or shape (r >= 1)");
  const int64_t w5 = (r + 5) / 6;
  for (int64_t row = 0; row < rows; ++row)
    for (int64_t k = 0; k < r; ++k) {
      const uint32_t f = (packed[row * w5 + k / 6] >> (5 * (k % 6))) & 31u;
      codes[row * r + k] = int8_t(f >= 16 ? int(f) - 32 : int(f));
    }
  return ARCHEAD_OK;
}

archead_status archead_pack_int4(const int8_t* codes, int64_t rows, int64_t d,
                                 uint8_t* packed) {
  if (!codes || !packed || rows < 0 || d <= 0 || d % 8)
    return fail(ARCHEAD_E_INVALID_ARG, "pack_int4: bad pointers or shape (d %% 8 == 0)");
  for (int64_t r = 0; r < rows; ++r) {
    const int8_t* c = codes + r * d;
    uint8_t* o = packed + r * (d / 2);
    for (int64_t w = 0; w < d / 8; ++w) {
      uint32_t q = 0;
      for (int k = 0; k < 8; ++k) {
        int v = c[8 * w + k];
        if (v < -8 || v > 7)
          return fail(ARCHEAD_E_INVALID_ARG, "pack_int4: code %d out of [-8, 7] at (%lld, %lld)",
                      v, (long long)r, (long long)(8 * w + k));
        // element 2j -> bits [4j, 4j+4), element 2j+1 -> bits [16+4j, 20+4j)
        int shift = 4 * (k >> 1) + ((k & 1) ? 16 : 0);
        q |= uint32_t(v + 8) << shift;
      }
      o[4 * w + 0] = uint8_t(q);
      o[4 * w + 1] = uint8_t(q >> 8);
      o[4 * w + 2] = uint8_t(q >> 16);
      o[4 * w + 3] = uint8_t(q >> 24);
    }
  }
  return ARCHEAD_OK;
}

archead_status archead_unpack_int4(const uint8_t* packed, int64_t rows, int64_t d,
                                   int8_t* codes) {
  if (!codes || !packed || rows < 0 || d <= 0 || d % 8)
    return fail(ARCHEAD_E_INVALID_ARG, "unpack_int4: bad pointers or shape (d %% 8 == 0)");
  for (int64_t r = 0; r < rows; ++r) {
    const uint8_t* p = packed + r * (d / 2);
    int8_t* c = codes + r * d;
    for (int64_t w = 0; w < d / 8; ++w) {
      uint32_t q = uint32_t(p[4 * w]) | uint32_t(p[4 * w + 1]) << 8 |
                   uint32_t(p[4 * w + 2]) << 16 | uint32_t(p[4 * w + 3]) << 24;
      for (int k = 0; k < 8; ++k) {
        int shift = 4 * (k >> 1) + ((k & 1) ? 16 : 0);
        c[8 * w + k] = int8_t(int((q >> shift) & 0xF) - 8);
      }
    }
  }
  return ARCHEAD_OK;
}

archead_status archead_set_gemv_max_m(archead_handle* h, int64_t m) {
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if (m < -1) return fail(ARCHEAD_E_INVALID_ARG, "gemv_max_m must be >= -1");
  h->gemv_max_m.store(m == -1 ? kDefaultGemvMaxM : m);
  return ARCHEAD_OK;
}

archead_status archead_set_launch(archead_handle* h, int knob, int64_t value) {
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  switch (knob) {
    case ARCHEAD_LAUNCH_GEMV_BLOCKS_PER_CU:
    case ARCHEAD_LAUNCH_GEMV_GRID:
    case ARCHEAD_LAUNCH_DEC_BLOCKS:
    case ARCHEAD_LAUNCH_MID_BLOCKS:
      if (value < 0 || value > (int64_t(1) << 30))
        return fail(ARCHEAD_E_INVALID_ARG, "launch size must be in [0, 2^30]");
      break;
    case ARCHEAD_LAUNCH_TILE_WAVES:
      if (value != 0 && value != 4 && value != 8)
        return fail(ARCHEAD_E_INVALID_ARG, "tile waves must be 0, 4 or 8");
      break;
    case ARCHEAD_LAUNCH_TILE_ROWS:
      if (value != 0 && value != 64 && value != 128)
        return fail(ARCHEAD_E_INVALID_ARG, "tile rows must be 0, 64 or 128");
      break;
    case ARCHEAD_LAUNCH_T_SPIN_LIMIT:
      if (value < -1 || value > (int64_t(1) << 30))
        return fail(ARCHEAD_E_INVALID_ARG, "spin limit must be in [-1, 2^30]");
      break;
    default:
      return fail(ARCHEAD_E_INVALID_ARG, "unknown launch knob");
  }
  h->launch[knob].store(value);
  // GEMV grids are cached per kernel variant: recompute them
  if (knob == ARCHEAD_LAUNCH_GEMV_BLOCKS_PER_CU || knob == ARCHEAD_LAUNCH_GEMV_GRID)
    for (auto& c : h->grid_cache) c.store(0);
  return ARCHEAD_OK;
}

archead_status archead_get_launch(const archead_handle* h, int knob, int64_t* value) {
  if (!h || !value) return fail(ARCHEAD_E_INVALID_ARG, "NULL argument");
  if (knob < 0 || knob >= ARCHEAD_LAUNCH_KNOBS) return fail(ARCHEAD_E_INVALID_ARG, "unknown launch knob");
  *value = h->launch[knob].load();
  return ARCHEAD_OK;
}

archead_status archead_set_timing_events(archead_handle* h, void* start, void* stop) {
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if ((start == nullptr) != (stop == nullptr))
    return fail(ARCHEAD_E_INVALID_ARG, "start and stop must both be set or both be NULL");
  h->ev_start.store(start);
  h->ev_stop.store(stop);
  return ARCHEAD_OK;
}

archead_status archead_set_dec_range(archead_handle* h, int64_t min_m, int64_t max_m) {
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if (min_m < -1 || max_m < -1) return fail(ARCHEAD_E_INVALID_ARG, "dec range bounds must be >= -1");
  int64_t r[4];
  default_ranges(h->desc, r);
  h->dec_min_m.store(min_m == -1 ? r[0] : min_m);
  h->dec_max_m.store(max_m == -1 ? r[1] : max_m);
  return ARCHEAD_OK;
}

archead_status archead_get_dec_range(const archead_handle* h, int64_t* min_m, int64_t* max_m) {
  if (!h || !min_m || !max_m) return fail(ARCHEAD_E_INVALID_ARG, "NULL argument");
  *min_m = h->dec_min_m.load();
  *max_m = h->dec_max_m.load();
  return ARCHEAD_OK;
}

archead_status archead_set_mid_range(archead_handle* h, int64_t min_m, int64_t max_m) {
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if (min_m < -1 || max_m < -1) return fail(ARCHEAD_E_INVALID_ARG, "mid range bounds must be >= -1");
  int64_t r[4];
  default_ranges(h->desc, r);
  h->mid_min_m.store(min_m == -1 ? r[2] : min_m);
  h->mid_max_m.store(max_m == -1 ? r[3] : max_m);
  return ARCHEAD_OK;
}

archead_status archead_get_mid_range(const archead_handle* h, int64_t* min_m, int64_t* max_m) {
  if (!h || !min_m || !max_m) return fail(ARCHEAD_E_INVALID_ARG, "NULL argument");
  *min_m = h->mid_min_m.load();
  *max_m = h->mid_max_m.load();
  return ARCHEAD_OK;
}

int64_t archead_get_gemv_max_m(const archead_handle* h) {
  return h ? h->gemv_max_m.load() : -1;
}

}  // extern "C"
