// Launcher of the decode products for a batch of sequences over the union
// of their retained sets (gemv_shared.hip).  Arguments are validated by the
// C-ABI layer (api.hip) before it is called.
#pragma once

#include "kernels.h"

namespace rmm {

// Decode products of B <= kShareMaxB sequences over the union of their sets
// (each kept weight row read once for all of them).  The contraction axis is
// cut into ranges of kShareRange indices; the layout function carves a
// group's workspace (pos, rows, cnt, xs, P) from ws (which may be null when
// only the size is wanted), sets R and chunks, and returns its bytes.
constexpr int kShareRange = 512;
constexpr int kShareMaxB = 32;
struct ShareGroup {
    const uint16_t *X;      // [B][ldx] bf16, one token per sequence
    const uint16_t *W;      // [K][ldw] bf16, 16-byte aligned, ldw % 8 == 0
    const int32_t *idx;     // [B][k] ascending lists
    uint16_t *Y;            // [B][ldy] bf16
    int32_t *pos;           // [B][R+1] list position of each range boundary
    int32_t *rows;          // [R][kShareRange] union rows of each range
    int32_t *cnt;           // [R] union size of each range
    uint16_t *xs;           // [R][32][kShareRange] activations over the union rows
    float *P;               // [B][R][N] fp32 partials when R > 1
    int N, K, k, R, chunks;
    int64_t ldx, ldw, ldy;
    int first_o, first_u, first_p, first_r;
};
struct ShareGroups {
    ShareGroup g[kMaxGemvGroups];
    int n;
};
size_t share_group_layout(int64_t B, int64_t N, int64_t K, void *ws, ShareGroup *q);
hipError_t launch_share_products(ShareGroups G, int64_t B, hipStream_t stream);

}  // namespace rmm
