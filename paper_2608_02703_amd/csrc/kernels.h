// Kernel entry points of the packed-head forward, one translation unit per
// kernel family: each selector returns the device function to launch (with
// hipExtLaunchKernel / hipLaunchKernel) for a variant.
#pragma once

namespace archead {
namespace kern {

// decode GEMV k_gemv<TOK, LPR, CE, SC8, GEN>: tok 1..4 tokens per pass, lpr
// lanes per vocabulary row (1, 2, 4, ..., 64), ce fused softmax, sc8 8-bit
// scales, gen the factor-code reads (0 aligned int8; 1 int8 of any rank; 2
// with ARCHEAD_I5 core-left codes; 1 and 2 only for lpr 8 and 16, else null)
const void* gemv(int tok, int lpr, bool ce, bool sc8, int gen);
// the single-token GEMV with the fused top-k epilogue (k_gemv<1, LPR, false,
// SC8, GEN, true>; null where gemv has no such variant), the top-k of rows
// of fp32 logits and the merge of per-partial top-k lists
const void* gemv_topk(int lpr, bool sc8, int gen);
const void* topk_rows();
const void* topk_merge(int block);   // k rounds; workgroups of 256 or kTopKMergeBlock threads, kTopKMergeC candidates each
const void* topk_merge_scan();   // any number of candidates
// MFMA decode kernel k_dec<GW, CE, EK, SC8, GEN>: gw = g / 32 code words per
// lane and group (1, 2, 4), ek expansion K-chunks held (2 or 4), gen as for
// gemv (every variant exists)
const void* dec(int gw, bool ce, int ek, bool sc8, int gen);
// several-token kernel k_mid: gw = g / 32 (2 or 4), gen as for dec
const void* mid(int gw, bool ce, bool sc8, int gen);
// tiled many-token kernel k_mfma<CE, TM, NW> (tm = 256 or 128 token rows
// per tile with nw = 8 waves per workgroup, or tm = 128 or 64 with nw = 4)
// and its prologue kernels
const void* mfma(bool ce, int tm, int nw);
// the tiled kernel's fidelity pass (xe = 1: dense rows streamed beside the
// packed codes) and rank pass (xe = 2), 64-row tiles of 4 waves, and the
// per-token merge of the fidelity pass's tile statistics
const void* mfma_fid(int xe);
const void* fid_head_merge();
const void* prep();
const void* stage1m();
const void* stage1m_fin();

}  // namespace kern
}  // namespace archead
