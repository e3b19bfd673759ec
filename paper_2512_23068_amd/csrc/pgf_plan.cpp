// Host-side planning of a libpgf call (see pgf_plan.h).
//
// Tiling.  Each (batch, channel) owns N independent recurrences.  One thread
// keeps nt of them in registers and ns = N/nt threads share a channel, so a
// sequence position costs one thread nt*(1+K) state updates.  When B*D*ns
// threads cannot fill the GPU, the sequence is cut into segments of `seg`
// steps that run in parallel: each segment is first scanned from a zero
// state (its end state and its sums of Delta and dDelta give the exact
// two-step composition of the augmented operator, Prop. 3.2 Eq. 5), a short
// sequential carry turns those into the true state entering every segment,
// and the segments are then rescanned from their true entry states while the
// outputs are written.  Host blocks of chunk_segs segments bound the
// workspace independently of L (the tiling of Alg. 1).
#include "pgf_plan.h"

#include <algorithm>

namespace pgf {

namespace {

constexpr int64_t kMaxSeg = 65536;
constexpr int kMaxChunkSegs = 4096;
// Scan blocks (256 threads) resident at once on an MI355X: 256 compute units
// x 4 blocks at the scan kernels' register use.  A launch whose block count
// is a multiple of this has no partly filled last round.
constexpr int64_t kResidentBlocks = 1024;
constexpr int64_t kSimds = 1024;
constexpr int64_t kDefaultSeg = 256;
constexpr int64_t kMaxChunkLen = int64_t(1) << 18;
// Workspace caps (of 288 GB of HBM): large enough that the benchmarked
// configurations of every order and variant run long sequences in one host
// block of whole rounds of resident blocks.
constexpr size_t kWorkspaceCap = size_t(512) << 20;
constexpr size_t kLaWorkspaceCap = size_t(1) << 30;
// A low-rank call also keeps Delta and dDelta_k of its host block: a larger cap keeps
// its host blocks as long as the others' (2 GiB of 288 GB).
constexpr size_t kLowRankWorkspaceCap = size_t(2) << 30;
constexpr int kMaxRank = 128;

int64_t gcd64(int64_t a, int64_t b) {
    while (b) {
        const int64_t t = a % b;
        a = b;
        b = t;
    }
    return a;
}

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

}  // namespace

int make_plan(const pgf_params *p, Plan *plan, size_t ws_cap) {
    if (!p || !plan) return PGF_ERR_INVALID_ARG;
    if (p->order < 0 || p->order > 3) return PGF_ERR_INVALID_ARG;
    const int order = p->order == 0 ? 1 : p->order;
    // The parameter flows carry two sensitivity states (dh/dA, dh/dB) and
    // need no tangent projections; n_dirs is not read.
    const int64_t B = p->batch, L = p->seqlen, D = p->d_inner, N = p->d_state;
    if (p->delta_flows < 0 || p->delta_flows > 1) return PGF_ERR_INVALID_ARG;
    if (p->delta_flows && order != 3) return PGF_ERR_INVALID_ARG;
    const int64_t K = order == 3 ? (p->delta_flows ? 4 : 2) : p->n_dirs;
    if (B < 1 || L < 0 || D < 1 || N < 1 || K < 1) return PGF_ERR_INVALID_ARG;
    if (p->in_dtype != PGF_F32 && p->in_dtype != PGF_BF16) return PGF_ERR_INVALID_ARG;
    if (!(N == 4 || N == 8 || N == 16 || N == 32 || N == 64)) return PGF_ERR_UNSUPPORTED;
    if (!(K == 1 || K == 2 || K == 4 || K == 8)) return PGF_ERR_UNSUPPORTED;
    // Guard the 64-bit index arithmetic of the kernels with a wide margin.
    if (B > 65535 || D > (int64_t(1) << 24) || L > (int64_t(1) << 40)) return PGF_ERR_UNSUPPORTED;
    if ((1 + K) * B * N * D > (int64_t(1) << 36)) return PGF_ERR_UNSUPPORTED;
    if ((double)K * B * (double)L * D > 9.0e18 / 16) return PGF_ERR_UNSUPPORTED;

    if (order == 2 && K != 2) return PGF_ERR_INVALID_ARG;
    if (p->drive < 0 || p->drive > 1 || p->activation < 0 || p->activation > 1) return PGF_ERR_INVALID_ARG;
    const int var = (p->drive == PGF_DRIVE_ZOH ? 1 : 0) |
                    ((p->activation != PGF_ACT_IDENTITY || p->D_res) ? 2 : 0);
    // the variants belong to the first order; the parameter flows also take
    // the ZOH drive and the output map
    if (var && order == 2) return PGF_ERR_UNSUPPORTED;
    const int cplx = p->A_im ? 1 : 0;
    if (var && !cplx && order != 3 && (K > 2 || N > 16)) return PGF_ERR_UNSUPPORTED;
    // the complex transition takes either drive, every N and K of the real
    // first order; the output map is applied to its real read-out
    if (cplx && order != 1) return PGF_ERR_UNSUPPORTED;
    if (p->n_groups < 0) return PGF_ERR_INVALID_ARG;
    const int64_t groups = p->n_groups > 1 ? p->n_groups : 1;
    if (groups > 1) {
        if (D % groups != 0 || (D / groups) % 64 != 0) return PGF_ERR_INVALID_ARG;
        if (order != 1 || cplx || (var & 1) || K > 2 || N > 16) return PGF_ERR_UNSUPPORTED;
        // one projection pass of 2*groups*N <= 128 columns, a power of two
        if (groups * N > 64 || !is_pow2(groups * N)) return PGF_ERR_UNSUPPORTED;
    }
    if (p->dt_rank < 0 || p->dt_rank > kMaxRank) return PGF_ERR_INVALID_ARG;
    const int rank = p->dt_rank;
    if (rank && (order != 1 || cplx || groups > 1 || (var & 1) || K > 2 || N > 16)) return PGF_ERR_UNSUPPORTED;

    Plan q{};
    q.B = B; q.L = L; q.D = D; q.N = N; q.K = K;
    q.order = order;
    q.var = var | (groups > 1 ? 4 : 0) | (rank ? 8 : 0);
    q.rank = rank;
    // the rank padded for the projection kernels: to a multiple of 16 up to
    // 64, of 32 above
    q.rc = rank <= 64 ? (rank + 15) / 16 * 16 : (rank + 31) / 32 * 32;
    q.groups = (int)groups;
    q.KP = order == 3 ? 0 : K;
    q.cplx = cplx;
    q.comp = (int)((1 + K + (order == 2 ? 1 : 0)) * (cplx ? 2 : 1));
    q.in_bf16 = p->in_dtype == PGF_BF16;
    // Registers per thread grow as nt*(3+K); keep them near 128.
    // (the parameter flows: up to 16 lanes per thread, N = 32 and 64 on
    // two and four threads)
    q.nt = (int)(order == 3 ? std::min<int64_t>(N, 16) : std::min<int64_t>(N, K >= 8 ? 4 : (K >= 4 ? 8 : 16)));
    q.ns = (int)(N / q.nt);
    q.R = (int)(groups * 2 * N * (1 + q.KP));
    // Wide f32 channel sums are cut into splits of at most about 2048
    // channels, so that a projection launch has enough blocks of moderate
    // length; bf16 rows (half the bytes, on the bf16 matrix cores) were
    // faster unsplit.
    q.ksplit = q.in_bf16 ? 1 : (int)std::min<int64_t>(4, (D + 2047) / 2048);
    q.dchunk = ((D + q.ksplit - 1) / q.ksplit + 31) / 32 * 32;

    // Blocks of one segment column (every channel, one segment).
    const int64_t nblk = B * ((D * q.ns + 255) / 256);
    int64_t seg;
    if (p->seg_len == -1) {
        seg = 0;
    } else if (p->seg_len != 0) {
        if (p->seg_len < 16 || p->seg_len > kMaxSeg || !is_pow2(p->seg_len)) return PGF_ERR_INVALID_ARG;
        seg = p->seg_len;
    } else {
        // Sequential when one segment column already gives every SIMD a wave
        // (a block is 4 waves; an MI355X has 1024 SIMDs).
        seg = (nblk * 4 >= kSimds) ? 0 : kDefaultSeg;
    }
    // Kernels address one host block with 32-bit element offsets.
    constexpr int64_t kMaxBlockElems = int64_t(1) << 30;
    int64_t cs;
    if (p->chunk_segs < 0 || p->chunk_segs > kMaxChunkSegs) return PGF_ERR_INVALID_ARG;
    const int64_t unit = seg ? seg : kSeqChunk;
    if (unit * D > kMaxBlockElems) return PGF_ERR_UNSUPPORTED;
    const int64_t cs_max = kMaxBlockElems / (unit * D);
    if (p->chunk_segs > cs_max) return PGF_ERR_INVALID_ARG;
    if (seg == 0) {
        cs = p->chunk_segs ? p->chunk_segs : 1;
        q.chunk_len = cs * kSeqChunk;
        q.chunk_segs = 1;
        cs = 1;
    } else if (p->chunk_segs) {
        cs = p->chunk_segs;
        q.chunk_len = cs * seg;
        q.chunk_segs = (int)cs;
    } else {
        // At least three rounds of resident blocks per launch, rounded to a
        // whole number of rounds when the workspace allows it.
        const size_t per_seg = (size_t)B * q.comp * (size_t)(N * D + D) * sizeof(float) +
                               (size_t)(1 + q.ksplit) * B * seg * q.R * sizeof(float) +
                               (size_t)(1 + K) * B * seg * (size_t)(rank ? q.rc + D : 0) * sizeof(float);
        const size_t wcap = ws_cap ? ws_cap : (rank ? kLowRankWorkspaceCap : kWorkspaceCap);
        const int64_t cap = std::max<int64_t>(1, (int64_t)(wcap / per_seg));
        const int64_t period = kResidentBlocks / gcd64(nblk, kResidentBlocks);
        const int64_t want = (3 * kResidentBlocks + nblk - 1) / nblk;
        cs = (want + period - 1) / period * period;
        if (cs > cap) cs = cap >= period ? cap / period * period : cap;
        cs = std::min<int64_t>(cs, kMaxChunkLen / seg);
        cs = std::min<int64_t>(std::min<int64_t>(cs, kMaxChunkSegs), cs_max);
        cs = std::max<int64_t>(cs, 1);
        q.chunk_len = cs * seg;
        q.chunk_segs = (int)cs;
    }
    q.seg = (int)seg;
    q.n_chunks = (L + q.chunk_len - 1) / q.chunk_len;

    const size_t f = sizeof(float);
    const size_t comp = (size_t)q.comp;
    Layout w{};
    size_t off = 0;
    w.state = off; off = align256(off + comp * B * N * D * f);
    w.bc = off;
    w.bc_half = align256((size_t)B * q.chunk_len * q.R * f);
    off += 2 * w.bc_half;
    w.part = off;
    off += (size_t)(q.ksplit - 1) * w.bc_half;
    if (seg) {
        const size_t G = (size_t)cs;
        w.agg_h = off;  off = align256(off + (size_t)B * G * comp * N * D * f);
        w.agg_s = off;  off = align256(off + (size_t)B * G * comp * D * f);
    } else {
        w.agg_h = w.agg_s = off;
    }
    w.gacc = off;
    if (order == 3) off = align256(off + (3 * (size_t)B * N * D + 3 * (size_t)B * D) * f);
    w.lr = off;
    if (rank) off = align256(off + (size_t)(1 + K) * B * q.chunk_len * q.rc * f);
    w.dt = off;
    if (rank) off = align256(off + (size_t)(1 + K) * B * q.chunk_len * D * f);
    w.total = off;
    q.ws = w;
    *plan = q;
    return PGF_OK;
}

int make_la_plan(const pgf_la_params *p, LaPlan *plan) {
    if (!p || !plan) return PGF_ERR_INVALID_ARG;
    const int64_t B = p->batch, H = p->heads, L = p->seqlen, DK = p->d_key, DV = p->d_value, K = p->n_dirs;
    if (B < 1 || H < 1 || L < 0 || DK < 1 || DV < 1 || K < 1) return PGF_ERR_INVALID_ARG;
    if (!(DK == 16 || DK == 32 || DK == 64)) return PGF_ERR_UNSUPPORTED;
    if (DV % 64 != 0 || DV > 4096) return PGF_ERR_UNSUPPORTED;
    if (K > 2) return PGF_ERR_UNSUPPORTED;
    if (B * H > (int64_t(1) << 20) || L > (int64_t(1) << 40)) return PGF_ERR_UNSUPPORTED;
    if ((double)K * B * H * (double)L * DV > 9.0e18 / 16) return PGF_ERR_UNSUPPORTED;
    LaPlan q{};
    q.B = B; q.H = H; q.L = L; q.DK = DK; q.DV = DV; q.K = K; q.BH = B * H;
    // Scan blocks of one segment column, counted in 256-thread units (a
    // block holds 64 value columns and DK/16 waves).
    const int64_t nblk = (q.BH * DV / 64 * (DK / 16) + 3) / 4;
    int64_t seg;
    if (p->seg_len == -1) {
        seg = 0;
    } else if (p->seg_len != 0) {
        if (p->seg_len < 16 || p->seg_len > kMaxSeg || !is_pow2(p->seg_len)) return PGF_ERR_INVALID_ARG;
        seg = p->seg_len;
    } else {
        seg = (nblk * 4 >= kSimds) ? 0 : 128;
    }
    if (p->chunk_segs < 0 || p->chunk_segs > kMaxChunkSegs) return PGF_ERR_INVALID_ARG;
    // Per-step offsets of one host block stay below 2^30 elements.
    constexpr int64_t kMaxBlockElems = int64_t(1) << 30;
    const int64_t unit = seg ? seg : kSeqChunk;
    if (unit * std::max(DK, DV) > kMaxBlockElems) return PGF_ERR_UNSUPPORTED;
    const size_t f = sizeof(float);
    int64_t cs;
    if (seg == 0) {
        cs = p->chunk_segs ? p->chunk_segs : 1;
        q.chunk_len = cs * kSeqChunk;
        q.chunk_segs = 1;
    } else if (p->chunk_segs) {
        cs = p->chunk_segs;
        q.chunk_len = cs * seg;
        q.chunk_segs = (int)cs;
    } else {
        // At least three rounds of resident blocks per launch, bounded by
        // a workspace cap of 1 GiB.
        const size_t per_seg = (size_t)q.BH * (1 + K) * ((size_t)DK * DV + DK) * f +
                               (size_t)q.BH * seg * (1 + K) * DK * f;
        const int64_t cap = std::max<int64_t>(1, (int64_t)(kLaWorkspaceCap / per_seg));
        cs = (3 * kResidentBlocks + nblk - 1) / nblk;
        cs = std::min<int64_t>(std::min<int64_t>(cs, cap), kMaxChunkSegs);
        cs = std::min<int64_t>(cs, kMaxChunkLen / seg);
        cs = std::max<int64_t>(cs, 1);
        q.chunk_len = cs * seg;
        q.chunk_segs = (int)cs;
    }
    if (q.chunk_len * std::max(DK, DV) > kMaxBlockElems) return PGF_ERR_INVALID_ARG;
    q.seg = (int)seg;
    q.n_chunks = (L + q.chunk_len - 1) / q.chunk_len;
    const size_t comp = (size_t)(1 + K);
    size_t off = 0;
    q.state = off; off = align256(off + comp * q.BH * DK * DV * f);
    q.rec = off;   off = align256(off + (size_t)q.BH * q.chunk_len * (1 + K) * DK * f);
    const size_t G = seg ? (size_t)q.chunk_segs : 1;
    q.agg_h = off; off = align256(off + (size_t)q.BH * G * comp * DK * DV * f);
    q.agg_s = off; off = align256(off + (size_t)q.BH * G * comp * DK * f);
    q.total = off;
    *plan = q;
    return PGF_OK;
}

}  // namespace pgf

extern "C" size_t pgf_la_workspace_bytes(const pgf_la_params *p) {
    pgf::LaPlan q;
    if (pgf::make_la_plan(p, &q) != PGF_OK) return 0;
    return q.total;
}

extern "C" int pgf_la_plan(const pgf_la_params *p, pgf_plan_info *info) {
    if (!info) return PGF_ERR_INVALID_ARG;
    pgf::LaPlan q;
    const int rc = pgf::make_la_plan(p, &q);
    if (rc != PGF_OK) return rc;
    info->n_per_thread = (int32_t)q.DK;
    info->n_split = 1;
    info->seg_len = q.seg;
    info->chunk_segs = q.chunk_segs;
    info->chunk_len = q.chunk_len;
    info->n_chunks = q.n_chunks;
    info->workspace_bytes = q.total;
    return PGF_OK;
}

extern "C" const char *pgf_status_string(int s) {
    switch (s) {
        case PGF_OK: return "PGF_OK";
        case PGF_ERR_INVALID_ARG: return "PGF_ERR_INVALID_ARG: invalid argument (NULL pointer, size or overlap)";
        case PGF_ERR_UNSUPPORTED: return "PGF_ERR_UNSUPPORTED: shape not supported (N in {4,8,16,32,64}, K in {1,2,4,8})";
        case PGF_ERR_WORKSPACE: return "PGF_ERR_WORKSPACE: workspace missing or smaller than pgf_workspace_bytes()";
        case PGF_ERR_HIP: return "PGF_ERR_HIP: a HIP runtime call or kernel launch failed";
        case PGF_ERR_SCRATCH:
            return "PGF_ERR_SCRATCH: the call needs more workspace than the static scratch of "
                   "pgf_scan_jvp_noalloc (PGF_SCRATCH_BYTES)";
        default: return "PGF: unknown status";
    }
}
