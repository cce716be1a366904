// Compile-time configuration of the bf16 MFMA sparse-attention kernel.
#pragma once

namespace relaxkv {

// Tile configuration of the bf16 MFMA attention kernel (compile-time; the
// defaults are the tuned MI355X configuration).
#ifndef RELAXKV_ATTN_WAVES
#define RELAXKV_ATTN_WAVES 8        // waves per workgroup
#endif
#ifndef RELAXKV_ATTN_TILE
#define RELAXKV_ATTN_TILE 128       // keys per LDS tile (double-buffered)
#endif
#ifndef RELAXKV_ATTN_SCHED
#define RELAXKV_ATTN_SCHED 1        // interleave K-fragment LDS reads with the QK^T MFMAs
#endif
#ifndef RELAXKV_ATTN_SETPRIO
#define RELAXKV_ATTN_SETPRIO 1      // raise wave priority during MFMA phases
#endif
#ifndef RELAXKV_ATTN_VPAD
#define RELAXKV_ATTN_VPAD 32        // V tile row padding (elements): conflict-free transposing reads
#endif
#ifndef RELAXKV_ATTN_ROWBLOCKS
#define RELAXKV_ATTN_ROWBLOCKS 1    // 32-row MFMA blocks per wave
#endif
// (target, head) rows per workgroup: a GQA group of G heads must fit.
constexpr int kAttnRows = RELAXKV_ATTN_WAVES * RELAXKV_ATTN_ROWBLOCKS * 32;

}  // namespace relaxkv
