// libpgf: decaying linear attention with its tangent flow (App. F: linear
// transformers, RetNet and RWKV-6 as general linear recurrences) for gfx950.
//
// The state of one (batch, head) is a dk x dv matrix S.  A block owns 64
// value columns of one head and splits the key dimension into slices of
// kKeys: a thread holds S[s*kKeys .. (s+1)*kKeys - 1, j .. j+kCols-1] (and
// the tangents) in registers, kKeys * kCols = 16 entries, so each key-side
// value it reads serves kCols columns (la_cols: 2 in the pass with outputs,
// 4 in the aggregate pass).  The lanes that share a slice need the same
// key-side values per step (q, k, alpha = exp(g), their tangents): the
// block stages them in LDS a tile of steps ahead and the lanes read them as
// broadcasts.  The per-lane inputs are v and dv_k of its columns; the
// partial outputs of a tile of steps are summed over the slices through LDS
// in a fixed order.
//
// Kernels, per host block of steps [t0, t0+len):
//   k_la_prep      alpha = exp(g) and alpha*dg_k per step into records, and
//                  the segment sums of g and dg_k
//   k_la_scan<false>  zero-start segment aggregates (end states)
//   k_la_carry     sequential over the block's segments, per lane: a segment
//                  maps (S, dS_k) to (P S + S0, P dS_k + Q_k S + dS0_k) with
//                  P = exp(sum g), Q_k = P sum dg_k (multiplications only)
//   k_la_scan<true>   rescan from the true entry states, writes o and do_k
// The sequential evaluation (enough columns to fill the GPU) runs k_la_prep
// and k_la_scan<true> only.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "pgf_exp.h"
#include "pgf_plan.h"
#include "pgf_timing.h"

namespace pgf {
namespace la {

constexpr int kThreads = 256;       // threads per block of the elementwise kernels
// Value columns per thread in the scan (the key dimensions per thread are
// 16 / columns, so a thread holds 16 entries of S): two in the pass with
// outputs, four in the aggregate pass, whose fewer fields per step leave
// room for the wider column block.
template <bool OUT>
constexpr int la_cols() { return OUT ? 2 : 4; }
constexpr float kLog2eHi = 1.44269502162933349609375f;  // log2(e) rounded to f32
constexpr float kLog2eLo = 1.925963033500011079e-08f;   // log2(e) - kLog2eHi
constexpr float kLn2 = 0.693147180559945309f;

// e^v within a few ulp for moderate |v|: v*log2(e) split into p + lo (an fma
// recovers the rounding of p), 2^p from the hardware exponential and
// 2^lo ~ 1 + lo*ln2 as a correction; lo also carries the lift that cancels
// the hardware exponential's mean bias near 1 (pgf_exp.h), since the decay
// alpha = e^g of a long-memory key is close to 1.
__device__ __forceinline__ float exp_acc(float v) {
    const float p = v * kLog2eHi;
    const float lo = fmaf(v, kLog2eHi, -p) + fmaf(v, kLog2eLo, kExp2Lift);
    const float e = __builtin_amdgcn_exp2f(p);
    return fmaf(e, lo * kLn2, e);
}

// ---------------------------------------------------------------- records
// Thread (segment g, key index i) of head bh, over the segment's steps:
//   rec[bh][t] = [alpha | alpha*dg_0 | ..]  (DK each), alpha = exp(g),
// and, when sums is set, the segment sums sums[bh][g][0][i] = sum_t g_t[i],
// sums[bh][g][1+k][i] = sum_t dg_k,t[i].  Reads and writes along i are
// coalesced.
template <int DK, int K>
__global__ __launch_bounds__(kThreads) void k_la_prep(
    const float *__restrict__ g, const float *__restrict__ dg, float *__restrict__ rec, float *__restrict__ sums,
    int64_t BH, int64_t L, int64_t t0, int64_t len, int64_t Tc, int64_t S, int G) {
    constexpr int SPB = kThreads / DK;   // segments per block
    constexpr int R = (1 + K) * DK;
    const int tid = threadIdx.x;
    const int i = tid % DK;
    const int gs = blockIdx.x * SPB + tid / DK;
    const int64_t bh = blockIdx.y;
    if (gs >= G) return;
    const int64_t ts = (int64_t)gs * S;
    const int64_t te = ts + S < len ? ts + S : len;
    const int64_t row0 = bh * L + t0;        // row of (bh, t0) in g
    const int64_t kst = BH * L;              // rows between tangent directions
    float *rb = rec + bh * Tc * R + i;
    float sg = 0.0f, sdg[K];
#pragma unroll
    for (int kk = 0; kk < K; ++kk) sdg[kk] = 0.0f;
#pragma unroll 4
    for (int64_t t = ts; t < te; ++t) {
        const float gv = g[(row0 + t) * DK + i];
        const float a = exp_acc(gv);
        sg += gv;
        float *r = rb + t * R;
        r[0] = a;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) {
            const float dgv = dg[(kk * kst + row0 + t) * DK + i];
            sdg[kk] += dgv;
            r[(1 + kk) * DK] = a * dgv;
        }
    }
    if (sums) {
        float *sb = sums + (bh * G + gs) * (1 + K) * DK + i;
        sb[0] = sg;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) sb[(1 + kk) * DK] = sdg[kk];
    }
}

// ---------------------------------------------------------------- scan
template <int DK, int K, bool OUT>
constexpr int la_fields() { return 2 + 2 * K + (OUT ? 1 + K : 0); }

template <int DK, int K, bool OUT>
__global__ __launch_bounds__(64 * (DK / 16)) __attribute__((amdgpu_waves_per_eu(K == 1 ? 4 : 2))) void k_la_scan(
    const float *__restrict__ q, const float *__restrict__ k, const float *__restrict__ v,
    const float *__restrict__ dq, const float *__restrict__ dk, const float *__restrict__ dv,
    const float *__restrict__ rec, const float *init, int64_t ibs, int64_t igs, int64_t ics,
    float *__restrict__ o, float *__restrict__ do_, float *end_state, float *__restrict__ agg_h,
    int64_t BH, int64_t L, int64_t DV, int64_t t0, int64_t len, int64_t Tc, int64_t S, int G) {
    constexpr int NW = DK / 16;
    constexpr int kCols = la_cols<OUT>();
    constexpr int kKeys = 16 / kCols;
    constexpr int NS = DK / kKeys;    // key slices (kCols per wave)
    constexpr int NTH = 64 * NW;
    constexpr int R = (1 + K) * DK;   // floats per step record
    constexpr int TT = OUT ? 4 : 2;   // steps per tile
    constexpr int F = la_fields<DK, K, OUT>();
    constexpr int FA = 2 + 2 * K;     // fields of the state update
    constexpr int NPF = (TT * F * DK + NTH - 1) / NTH;   // key-side floats per thread and tile
    __shared__ float kvs[2][TT][F][DK];
    __shared__ float red[OUT ? 2 : 1][TT][1 + K][NS][64];

    const int tid = threadIdx.x;
    const int lane = tid % 64;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64);
    const int64_t groups = DV / 64;
    const int64_t bh = blockIdx.x / groups;
    const int64_t jg = (blockIdx.x % groups) * 64;   // first column of the block
    constexpr int LPS = 64 / kCols;                   // lanes per key slice
    const int64_t j = jg + kCols * (lane % LPS);      // this thread's columns j .. j+kCols-1
    const int g = blockIdx.y;
    const int64_t ts = (int64_t)g * S;
    const int64_t te = ts + S < len ? ts + S : len;
    if (ts >= te) return;   // uniform over the block
    const int sl = kCols * w + lane / LPS;            // key slice
    const int i0 = sl * kKeys;

    float Sm[kKeys][kCols], dS[K][kKeys][kCols];
    if constexpr (OUT) {
        const float *ib = init + bh * ibs + g * igs + (int64_t)i0 * DV + j;
#pragma unroll
        for (int i = 0; i < kKeys; ++i) {
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                Sm[i][c] = ib[i * DV + c];
#pragma unroll
                for (int kk = 0; kk < K; ++kk) dS[kk][i][c] = ib[(1 + kk) * ics + i * DV + c];
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < kKeys; ++i) {
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                Sm[i][c] = 0.0f;
#pragma unroll
                for (int kk = 0; kk < K; ++kk) dS[kk][i][c] = 0.0f;
            }
        }
    }

    const int64_t kst = BH * L;                       // rows between tangent directions
    const int64_t row0 = bh * L + t0;
    const float *rb = rec + bh * Tc * R;
    const float *vb = v + row0 * DV + j;

    // The key-side data of a tile is TT*F rows of DK floats (row r = step
    // jj*F + field f); thread tid loads element tid % DK of the rows
    // r = tid / DK (mod RPI), so every row is one coalesced load and the
    // field of each load is known at compile time.  Loads past the segment
    // repeat its last step.  In the pass with outputs, those steps are
    // staged as neutral data (alpha = 1, every other field 0): such a step
    // leaves S and dS exactly as they are, so whole tiles run without a
    // per-step guard (their outputs are never written); the aggregate pass
    // skips them.
    constexpr int RPI = NTH / DK;          // rows covered by one pass of the block
    const int myrow = tid / DK, ki_ = tid % DK;
    auto key_row = [&](int f, int64_t t) -> const float * {
        if (f == 0) return rb + t * R;
        if (f == 1) return k + (row0 + t) * DK;
        if (f < FA) {
            const int kk = (f - 2) / 2;
            return (f % 2 == 0) ? rb + t * R + (1 + kk) * DK : dk + (kk * kst + row0 + t) * DK;
        }
        if (f == FA) return q + (row0 + t) * DK;
        return dq + ((f - FA - 1) * kst + row0 + t) * DK;
    };
    auto fetch = [&](int64_t tb, float *pre) {
#pragma unroll
        for (int r = 0; r < TT * F; ++r) {
            if (r % RPI == myrow) {
                const int jj = r / F, f = r % F;
                const int64_t t = tb + jj < te ? tb + jj : te - 1;
                pre[r / RPI] = key_row(f, t)[ki_];
            }
        }
    };
    auto stash = [&](int b, int64_t tb, const float *pre) {
#pragma unroll
        for (int r = 0; r < TT * F; ++r) {
            if (r % RPI == myrow) {
                const int f = r % F;
                float val = pre[r / RPI];
                if constexpr (OUT) val = tb + r / F < te ? val : (f == 0 ? 1.0f : 0.0f);
                kvs[b][r / F][f][ki_] = val;
            }
        }
    };

    // One step (tile slot jj) for this thread's key slice and kCols columns:
    // the state update, then the partial outputs summed over the slice.
    // part[c][0] = o, part[c][1+k] = do_k of column j + c.
    auto step = [&](int b, int jj, const float *vv, const float (*dvv)[kCols], float (*part)[1 + K]) {
        const float *rr = &kvs[b][jj][0][i0];
#pragma unroll
        for (int i = 0; i < kKeys; ++i) {
            const float a = rr[i], ki = rr[DK + i];
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                // the tangents read the old S; the two passes order the
                // updates differently (same values), whichever schedules
                // better
                if constexpr (OUT) {
#pragma unroll
                    for (int kk = 0; kk < K; ++kk) {
                        const float adg = rr[(2 + 2 * kk) * DK + i];
                        const float dki = rr[(3 + 2 * kk) * DK + i];
                        dS[kk][i][c] =
                            fmaf(a, dS[kk][i][c], fmaf(adg, Sm[i][c], fmaf(dki, vv[c], ki * dvv[kk][c])));
                    }
                    Sm[i][c] = fmaf(ki, vv[c], a * Sm[i][c]);
                } else {
                    const float sn = fmaf(ki, vv[c], a * Sm[i][c]);
#pragma unroll
                    for (int kk = 0; kk < K; ++kk) {
                        const float adg = rr[(2 + 2 * kk) * DK + i];
                        const float dki = rr[(3 + 2 * kk) * DK + i];
                        dS[kk][i][c] =
                            fmaf(a, dS[kk][i][c], fmaf(adg, Sm[i][c], fmaf(dki, vv[c], ki * dvv[kk][c])));
                    }
                    Sm[i][c] = sn;
                }
            }
        }
        if constexpr (OUT) {
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                float ov = 0.0f, dov[K];
#pragma unroll
                for (int kk = 0; kk < K; ++kk) dov[kk] = 0.0f;
#pragma unroll
                for (int i = 0; i < kKeys; ++i) {
                    const float qi = rr[FA * DK + i];
                    ov = fmaf(qi, Sm[i][c], ov);
#pragma unroll
                    for (int kk = 0; kk < K; ++kk)
                        dov[kk] = fmaf(rr[(FA + 1 + kk) * DK + i], Sm[i][c], fmaf(qi, dS[kk][i][c], dov[kk]));
                }
                part[c][0] = ov;
#pragma unroll
                for (int kk = 0; kk < K; ++kk) part[c][1 + kk] = dov[kk];
            }
        }
    };
    auto load_vdv = [&](int64_t t, float *vv, float (*dvv)[kCols]) {
#pragma unroll
        for (int c = 0; c < kCols; ++c) {
            vv[c] = vb[t * DV + c];
#pragma unroll
            for (int kk = 0; kk < K; ++kk) dvv[kk][c] = dv[(kk * kst + row0 + t) * DV + j + c];
        }
    };

    // Tiles of TT steps (the last one partial); the next tile's key-side data
    // and v, dv are in flight while a tile computes.  Every trip of the tile
    // loop is taken by the whole block.
    float pre[NPF];
    fetch(ts, pre);
    stash(0, ts, pre);
    float vc[TT][kCols], dvc[TT][K][kCols];
#pragma unroll
    for (int jj = 0; jj < TT; ++jj) load_vdv(ts + jj < te ? ts + jj : te - 1, vc[jj], dvc[jj]);
    __syncthreads();
    int buf = 0;
    for (int64_t tb = ts; tb < te; tb += TT) {
        const bool more = tb + TT < te;
        if (more) fetch(tb + TT, pre);
        float vn[TT][kCols], dvn[TT][K][kCols];
#pragma unroll
        for (int jj = 0; jj < TT; ++jj) {
            const int64_t t = tb + TT + jj < te ? tb + TT + jj : te - 1;
            load_vdv(t, vn[jj], dvn[jj]);
        }
        float part[TT][kCols][1 + K];
        if constexpr (OUT) {
#pragma unroll
            for (int jj = 0; jj < TT; ++jj) step(buf, jj, vc[jj], dvc[jj], part[jj]);
        } else {
            // (measured: the aggregate pass runs faster with the guard)
#pragma unroll
            for (int jj = 0; jj < TT; ++jj)
                if (tb + jj < te) step(buf, jj, vc[jj], dvc[jj], part[jj]);
        }
        if constexpr (OUT) {
#pragma unroll
            for (int jj = 0; jj < TT; ++jj)
#pragma unroll
                for (int c = 0; c <= K; ++c)
#pragma unroll
                    for (int e = 0; e < kCols; ++e) red[buf][jj][c][sl][kCols * (lane % LPS) + e] = part[jj][e][c];
        }
        if (more) stash(buf ^ 1, tb + TT, pre);
        __syncthreads();
        if constexpr (OUT) {
            // wave w completes steps jj = w, w + NW, ... of the tile, lane =
            // column jg + lane
            for (int jj = w; jj < TT; jj += NW) {
                const int64_t t = tb + jj;
                if (t >= te) break;
#pragma unroll
                for (int c = 0; c <= K; ++c) {
                    float acc = red[buf][jj][c][0][lane];
#pragma unroll
                    for (int s2 = 1; s2 < NS; ++s2) acc += red[buf][jj][c][s2][lane];
                    if (c == 0) o[(row0 + t) * DV + jg + lane] = acc;
                    else do_[((c - 1) * kst + row0 + t) * DV + jg + lane] = acc;
                }
            }
        }
        buf ^= 1;
#pragma unroll
        for (int jj = 0; jj < TT; ++jj)
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                vc[jj][c] = vn[jj][c];
#pragma unroll
                for (int kk = 0; kk < K; ++kk) dvc[jj][kk][c] = dvn[jj][kk][c];
            }
    }

    if constexpr (OUT) {
        if (end_state) {
            float *eb = end_state + bh * ibs + (int64_t)i0 * DV + j;
#pragma unroll
            for (int i = 0; i < kKeys; ++i)
#pragma unroll
                for (int c = 0; c < kCols; ++c) {
                    eb[i * DV + c] = Sm[i][c];
#pragma unroll
                    for (int kk = 0; kk < K; ++kk) eb[(1 + kk) * ics + i * DV + c] = dS[kk][i][c];
                }
        }
    } else {
        float *ab = agg_h + (bh * G + g) * (1 + K) * DK * DV + (int64_t)i0 * DV + j;
#pragma unroll
        for (int i = 0; i < kKeys; ++i)
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                ab[i * DV + c] = Sm[i][c];
#pragma unroll
                for (int kk = 0; kk < K; ++kk) ab[((1 + kk) * DK + i) * DV + c] = dS[kk][i][c];
            }
    }
}

// ---------------------------------------------------------------- carry
// One thread per lane (bh, i, j), sequential over the block's segments.
// state [(1+K)][BH][DK][DV] enters and leaves; seg [BH][G][(1+K)][DK][DV]
// holds each segment's zero-start end state on entry and is overwritten with
// the true state entering the segment.  sums [BH][G][(1+K)][DK] as written
// by k_la_prep.
template <int K>
__global__ __launch_bounds__(kThreads) void k_la_carry(
    float *__restrict__ seg, const float *__restrict__ sums, float *__restrict__ state, int64_t BH, int64_t DK,
    int64_t DV, int G) {
    constexpr int GB = K == 1 ? 16 : 8;
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t per = DK * DV;
    if (idx >= BH * per) return;
    const int64_t bh = idx / per, r = idx % per, i = r / DV;
    const int64_t cs = BH * per;
    float s = state[idx], ds[K];
#pragma unroll
    for (int kk = 0; kk < K; ++kk) ds[kk] = state[(1 + kk) * cs + idx];
    for (int g0 = 0; g0 < G; g0 += GB) {
        float e0[GB], e1[K][GB], sg[GB], sdg[K][GB];
#pragma unroll
        for (int jj = 0; jj < GB; ++jj) {
            const int g = g0 + jj < G ? g0 + jj : G - 1;
            const int64_t base = (bh * G + g) * (1 + K);
            e0[jj] = seg[base * per + r];
            sg[jj] = sums[base * DK + i];
#pragma unroll
            for (int kk = 0; kk < K; ++kk) {
                e1[kk][jj] = seg[(base + 1 + kk) * per + r];
                sdg[kk][jj] = sums[(base + 1 + kk) * DK + i];
            }
        }
#pragma unroll
        for (int jj = 0; jj < GB; ++jj) {
            if (g0 + jj >= G) break;
            const int64_t base = (bh * G + g0 + jj) * (1 + K);
            seg[base * per + r] = s;
#pragma unroll
            for (int kk = 0; kk < K; ++kk) seg[(base + 1 + kk) * per + r] = ds[kk];
            const float P = exp_series(sg[jj]);
#pragma unroll
            for (int kk = 0; kk < K; ++kk) ds[kk] = fmaf(P, ds[kk], fmaf(P * sdg[kk][jj], s, e1[kk][jj]));
            s = fmaf(P, s, e0[jj]);
        }
    }
    state[idx] = s;
#pragma unroll
    for (int kk = 0; kk < K; ++kk) state[(1 + kk) * cs + idx] = ds[kk];
}

// ---------------------------------------------------------------- state in/out
// dst[i] = src ? src[i] : 0 over n floats (the state layout is the ABI's).
__global__ __launch_bounds__(kThreads) void k_la_copy(const float *__restrict__ src, float *__restrict__ dst,
                                                      int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) dst[i] = src ? src[i] : 0.0f;
}

// ---------------------------------------------------------------- dispatch
struct LaLauncher {
    const LaPlan &q;
    const pgf_la_params &p;
    const float *qv, *kv, *vv, *gv, *dqv, *dkv, *dvv, *dgv;
    float *o, *dov;
    hipStream_t st;
    char *ws;

    float *state() const { return (float *)(ws + q.state); }
    float *rec() const { return (float *)(ws + q.rec); }
    float *agg_h() const { return (float *)(ws + q.agg_h); }
    float *agg_s() const { return (float *)(ws + q.agg_s); }

    template <int DK, int K>
    void block(int64_t t0, int64_t len) {
        const int64_t ND = DK * q.DV;
        const unsigned gx = (unsigned)(q.BH * q.DV / 64);
        const dim3 blk(64 * (DK / 16));
        const int64_t S = q.seg ? q.seg : len;
        const int G = (int)((len + S - 1) / S);
        {
            constexpr int SPB = kThreads / DK;
            Timed tm(0, st);
            hipLaunchKernelGGL((k_la_prep<DK, K>), dim3((unsigned)((G + SPB - 1) / SPB), (unsigned)q.BH),
                               dim3(kThreads), 0, st, gv, dgv, rec(), q.seg ? agg_s() : (float *)nullptr, q.BH, q.L,
                               t0, len, q.chunk_len, S, G);
        }
        if (q.seg == 0) {
            Timed tm(3, st);
            hipLaunchKernelGGL((k_la_scan<DK, K, true>), dim3(gx, 1), blk, 0, st, qv, kv, vv, dqv, dkv, dvv,
                               (const float *)rec(), (const float *)state(), ND, (int64_t)0, q.BH * ND, o, dov,
                               state(), (float *)nullptr, q.BH, q.L, q.DV, t0, len, q.chunk_len, len, 1);
            return;
        }
        {
            Timed tm(1, st);
            hipLaunchKernelGGL((k_la_scan<DK, K, false>), dim3(gx, (unsigned)G), blk, 0, st, qv, kv, vv, dqv, dkv,
                               dvv, (const float *)rec(), (const float *)nullptr, (int64_t)0, (int64_t)0, (int64_t)0,
                               o, dov, (float *)nullptr, agg_h(), q.BH, q.L, q.DV, t0, len, q.chunk_len, S, G);
        }
        {
            const int64_t lanes = q.BH * ND;
            Timed tm(2, st);
            hipLaunchKernelGGL((k_la_carry<K>), dim3((unsigned)((lanes + kThreads - 1) / kThreads)), dim3(kThreads),
                               0, st, agg_h(), (const float *)agg_s(), state(), q.BH, (int64_t)DK, q.DV, G);
        }
        {
            Timed tm(3, st);
            hipLaunchKernelGGL((k_la_scan<DK, K, true>), dim3(gx, (unsigned)G), blk, 0, st, qv, kv, vv, dqv, dkv,
                               dvv, (const float *)rec(), (const float *)agg_h(), (int64_t)G * (1 + K) * ND,
                               (int64_t)(1 + K) * ND, ND, o, dov, (float *)nullptr, (float *)nullptr, q.BH, q.L, q.DV,
                               t0, len, q.chunk_len, S, G);
        }
    }

    template <int DK, int K>
    int run_t() {
        const int64_t nst = q.BH * DK * q.DV;   // floats per state component
        const unsigned gs = (unsigned)((nst + kThreads - 1) / kThreads);
        {
            Timed tm(4, st);
            hipLaunchKernelGGL(k_la_copy, dim3(gs), dim3(kThreads), 0, st, p.S_in, state(), nst);
            for (int kk = 0; kk < K; ++kk)
                hipLaunchKernelGGL(k_la_copy, dim3(gs), dim3(kThreads), 0, st,
                                   p.dS_in ? p.dS_in + kk * nst : (const float *)nullptr, state() + (1 + kk) * nst,
                                   nst);
        }
        for (int64_t t0 = 0; t0 < q.L; t0 += q.chunk_len) {
            const int64_t len = q.L - t0 < q.chunk_len ? q.L - t0 : q.chunk_len;
            block<DK, K>(t0, len);
        }
        if (p.S_out || p.dS_out) {
            Timed tm(4, st);
            if (p.S_out)
                hipLaunchKernelGGL(k_la_copy, dim3(gs), dim3(kThreads), 0, st, (const float *)state(), p.S_out, nst);
            if (p.dS_out)
                hipLaunchKernelGGL(k_la_copy, dim3((unsigned)((K * nst + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                                   st, (const float *)(state() + nst), p.dS_out, K * nst);
        }
        return hipGetLastError() == hipSuccess ? PGF_OK : PGF_ERR_HIP;
    }

    int run() {
        switch (q.DK * 10 + q.K) {
            case 161: return run_t<16, 1>();
            case 162: return run_t<16, 2>();
            case 321: return run_t<32, 1>();
            case 322: return run_t<32, 2>();
            case 641: return run_t<64, 1>();
            case 642: return run_t<64, 2>();
            default: return PGF_ERR_UNSUPPORTED;
        }
    }
};

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
    return na && nb && pa < pb + nb && pb < pa + na;
}

}  // namespace la
}  // namespace pgf

extern "C" int pgf_la_scan_jvp(const float *q, const float *k, const float *v, const float *g, const float *dq,
                               const float *dk, const float *dv, const float *dg, const pgf_la_params *p, float *o,
                               float *do_, void *stream) {
    using namespace pgf;
    LaPlan pl;
    const int rc = make_la_plan(p, &pl);
    if (rc != PGF_OK) return rc;
    if (!p->workspace || p->workspace_bytes < pl.total || ((uintptr_t)p->workspace & 255))
        return PGF_ERR_WORKSPACE;
    if (pl.L > 0) {
        if (!q || !k || !v || !g || !dq || !dk || !dv || !dg || !o || !do_) return PGF_ERR_INVALID_ARG;
        const size_t f = sizeof(float);
        const size_t nk = (size_t)pl.BH * pl.L * pl.DK * f, nv = (size_t)pl.BH * pl.L * pl.DV * f;
        const void *ins[8] = {q, k, v, g, dq, dk, dv, dg};
        const size_t sz[8] = {nk, nk, nv, nk, nk * pl.K, nk * pl.K, nv * pl.K, nk * pl.K};
        for (int i = 0; i < 8; ++i)
            if (la::overlap(o, nv, ins[i], sz[i]) || la::overlap(do_, nv * pl.K, ins[i], sz[i]) ||
                la::overlap(p->workspace, pl.total, ins[i], sz[i]))
                return PGF_ERR_INVALID_ARG;
        if (la::overlap(o, nv, do_, nv * pl.K) || la::overlap(o, nv, p->workspace, pl.total) ||
            la::overlap(do_, nv * pl.K, p->workspace, pl.total))
            return PGF_ERR_INVALID_ARG;
    }
    (void)hipGetLastError();
    la::LaLauncher l{pl, *p, q, k, v, g, dq, dk, dv, dg, o, do_, (hipStream_t)stream, (char *)p->workspace};
    return l.run();
}
