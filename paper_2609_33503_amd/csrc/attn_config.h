// Compile-time configuration of the bf16 MFMA sparse-attention kernel.
#pragma once

namespace relaxkv {

// Defaults are the tuned MI355X configuration.
#ifndef RELAXKV_ATTN_WAVES
#define RELAXKV_ATTN_WAVES 12       // waves (32 rows each) per workgroup; one workgroup per CU
#endif
#ifndef RELAXKV_ATTN_KAHEAD
#define RELAXKV_ATTN_KAHEAD 4       // K fragments read from LDS ahead of their MFMA
#endif
#ifndef RELAXKV_ATTN_SCHED
#define RELAXKV_ATTN_SCHED 1        // interleave K-fragment LDS reads with the QK^T MFMAs
#endif
#ifndef RELAXKV_ATTN_SETPRIO
#define RELAXKV_ATTN_SETPRIO 0      // raise wave priority during MFMA phases
#endif
#ifndef RELAXKV_ATTN_LEAN
#define RELAXKV_ATTN_LEAN 1         // 3-input max chains and bf16 dot2 row sums in the softmax
#endif
// (target, head) rows per workgroup (the bf16 path takes GQA groups of at most
// this many heads, which keeps its row counts below 2^31).
constexpr int kAttnRows = RELAXKV_ATTN_WAVES * 32;

}  // namespace relaxkv
