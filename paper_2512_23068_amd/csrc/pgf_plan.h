// Host-side planning of a libpgf call: argument checks, tiling choice and
// workspace layout.  Plain C++ with no device access (the sanitizer tests
// build it with g++); shared by the launch code and by the host-only entry
// points (pgf_workspace_bytes, pgf_plan, pgf_la_*).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/pgf.h"

namespace pgf {

// Steps per unit of a sequential host block (a block is chunk_segs units).
// The parameter flows add their gradient partials to the running sums once
// per unit, so the order of those additions does not depend on the blocks.
constexpr int64_t kSeqChunk = 4096;

// Offsets (bytes) of the workspace sections; each is 256-byte aligned.
//   state   [(1+K)][B][N][D]         state carried between host blocks
//   bc      [2][B][Tc][R]            per-step projections of two host blocks
//                                    (the one being scanned and the next),
//                                    per group 2N(1+KP): B, dB_0..dB_{KP-1}, C, dC_0..
//   part    [S-1][B][Tc][R]          partial projections of channel splits 1..S-1
//   agg_h   [B][G][(1+K)][N][D]      segment end states from a zero start,
//                                    then (in place) the true state
//                                    entering each segment
//   agg_s   [B][G][(1+K)][D]         segment sums of Delta and dDelta_k
//   gacc    [3][B][N][D] + [3][B][D] parameter flows only: running gradient
//                                    sums (A, B offset, C offset) of the call,
//                                    then the per-channel ones (D_res,
//                                    w_delta, b_delta)
//   lr      [(1+K)][B][Tc][RC]       low rank only: x W_dx and dx_k W_dx, the
//                                    rank padded to RC (zero columns)
//   dt      [(1+K)][B][Tc][D]        low rank only: Delta and dDelta_k
// In the parameter flows K = 2 (the states dh/dA and dh/dB; 4 with the
// step size's dh/dw_delta and dh/db_delta) and agg_h also receives each
// segment's gradient partials after its rescan.
struct Layout {
    size_t state, bc, bc_half, part, agg_h, agg_s, gacc, lr, dt, total;   // bc_half: bytes of one bc buffer
};

struct Plan {
    int64_t B, L, D, N, K;
    int order;           // 1, 2, or 3 (parameter flows)
    int64_t KP;          // directions projected by k_proj (K, or 0 for order 3)
    int var;             // model variant bits of the first-order scan (kZoh 1, kOutMap 2, kGroups 4, kLowRank 8)
    int rank, rc;        // low-rank step size: rank R and its padded width (0 when off)
    int groups;          // channel groups with their own B and C (1 = one group)
    int cplx;            // complex diagonal transition (state in real/imaginary planes)
    int comp;            // state planes per lane: 1 + K (+ 1 for the mixed flow), twice that if complex
    int in_bf16;
    int nt, ns;          // states per thread, threads per channel (nt*ns == N)
    int seg;             // segment length; 0 = sequential evaluation
    int chunk_segs;      // segments per host block (1 when sequential)
    int64_t chunk_len;   // steps per host block
    int64_t n_chunks;
    int R;               // floats per step in bc: groups * 2N(1+KP)
    int ksplit;          // channel splits S of the projections (1 up to 2048 channels)
    int64_t dchunk;      // channels per split, a multiple of 32
    int noalloc;         // 1: run every host block in order on the caller's stream
                         // (no helper stream) and record no timing events
    Layout ws;
};

// Validates the size fields and fills *plan.  ws_cap bounds the workspace
// that the default host-block size may take (0: the library's caps); an
// explicit chunk_segs is not bounded.  Returns PGF_OK or an error.
int make_plan(const pgf_params *p, Plan *plan, size_t ws_cap = 0);

// Decaying linear attention.  Workspace sections (256-byte aligned):
//   state [(1+K)][BH][DK][DV]      state carried between host blocks (the
//                                  layout of S and dS in the ABI)
//   rec   [BH][Tc][(1+K)][DK]      per-step alpha = exp(g) and alpha*dg_k
//   agg_h [BH][G][(1+K)][DK][DV]   segment end states from a zero start,
//                                  then (in place) the true entry states
//   agg_s [BH][G][(1+K)][DK]       segment sums of g and dg_k
struct LaPlan {
    int64_t B, H, L, DK, DV, K, BH;
    int seg;             // segment length; 0 = sequential evaluation
    int chunk_segs;
    int64_t chunk_len, n_chunks;
    size_t state, rec, agg_h, agg_s, total;
};

int make_la_plan(const pgf_la_params *p, LaPlan *plan);

}  // namespace pgf
