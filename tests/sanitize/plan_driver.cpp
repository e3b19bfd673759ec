// Drives the host planner of libpgf (make_plan, make_la_plan,
// pgf_status_string; plain C++, no device) over a grid of valid and invalid
// arguments, for a build with AddressSanitizer and UndefinedBehaviorSanitizer.
// Besides running every path under the sanitizers it checks the layout of
// each accepted plan: sections in order, 256-byte aligned, inside the total,
// and a workspace that does not depend on the sequence length.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <initializer_list>

#include "../../paper_2512_23068_amd/csrc/pgf_plan.h"

static int failures = 0;

#define CHECK(cond)                                                                        \
    do {                                                                                   \
        if (!(cond)) {                                                                     \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond);             \
            ++failures;                                                                    \
        }                                                                                  \
    } while (0)

static void check_layout(const pgf::Plan &q) {
    const pgf::Layout &w = q.ws;
    const size_t offs[] = {w.state, w.bc, w.part, w.agg_h, w.agg_s, w.gacc, w.lr, w.dt, w.total};
    for (size_t i = 0; i < sizeof(offs) / sizeof(offs[0]); ++i) {
        CHECK(offs[i] % 256 == 0);
        if (i) CHECK(offs[i] >= offs[i - 1]);
    }
    CHECK(w.bc + 2 * w.bc_half <= w.part);
    CHECK(q.nt * q.ns == q.N);
    CHECK(q.n_chunks * q.chunk_len >= q.L);
    CHECK(q.L == 0 || (q.n_chunks - 1) * q.chunk_len < q.L);
    CHECK(q.chunk_len * q.D <= (int64_t(1) << 30));
    if (q.order == 3) {
        // up to 16 lanes per thread (N = 32, 64 on two, four), five planes with the
        // step size's flows, and room for the [3][B][N][D] + [3][B][D] sums
        CHECK(q.nt * q.ns == q.N && q.nt <= 16 && (q.K == 2 || q.K == 4) && q.comp == 1 + q.K);
        CHECK(w.lr - w.gacc >= (size_t)(3 * q.B * q.N * q.D + 3 * q.B * q.D) * sizeof(float));
    }
}

int main() {
    long plans = 0, rejected = 0;
    const int64_t Ns[] = {1, 4, 8, 12, 16, 32, 64, 128};
    const int64_t Ks[] = {0, 1, 2, 3, 4, 8, 9};
    const int64_t Ds[] = {1, 64, 77, 1536, 5120};
    const int segs[] = {0, -1, 16, 64, 100, 256, 1 << 17};
    for (int order = -1; order <= 4; ++order)
        for (int64_t N : Ns)
            for (int64_t K : Ks)
                for (int64_t D : Ds)
                    for (int seg : segs)
                        for (int dt = 0; dt < 3; ++dt)
                            for (int var = 0; var < 8; ++var) {
                                pgf_params p;
                                memset(&p, 0, sizeof(p));
                                p.batch = (D == 77) ? 3 : 1;
                                p.seqlen = 131072;
                                p.d_inner = D;
                                p.d_state = N;
                                p.n_dirs = K;
                                p.in_dtype = dt;
                                p.seg_len = seg;
                                p.order = order;
                                p.drive = var == 1;
                                p.activation = var == 2 ? 1 : (var == 5 ? 7 : 0);
                                p.A_im = var == 3 ? (const float *)16 : nullptr;   // tested for NULL only
                                p.n_groups = var == 4 ? 2 : 0;
                                p.dt_rank = (var == 5) ? 48 : 0;
                                // the step size's parameter flows, alone and with the ZOH drive
                                p.delta_flows = var >= 6 ? 1 : 0;
                                if (var == 7) p.drive = 1;
                                pgf::Plan q;
                                const int rc = pgf::make_plan(&p, &q);
                                CHECK(rc == PGF_OK || rc == PGF_ERR_INVALID_ARG || rc == PGF_ERR_UNSUPPORTED);
                                if (rc != PGF_OK) {
                                    ++rejected;
                                    continue;
                                }
                                ++plans;
                                check_layout(q);
                                // the workspace does not depend on L
                                for (int64_t L : {int64_t(0), int64_t(1), int64_t(8191), int64_t(1) << 24}) {
                                    pgf_params p2 = p;
                                    p2.seqlen = L;
                                    pgf::Plan q2;
                                    CHECK(pgf::make_plan(&p2, &q2) == PGF_OK);
                                    CHECK(q2.ws.total == q.ws.total);
                                }
                                // a smaller cap never gives a larger workspace
                                pgf::Plan q3;
                                if (pgf::make_plan(&p, &q3, size_t(64) << 20) == PGF_OK) {
                                    CHECK(q3.ws.total <= q.ws.total);
                                    check_layout(q3);
                                }
                            }
    // invalid pointers and extreme sizes are rejected, never used
    pgf::Plan q;
    CHECK(pgf::make_plan(nullptr, &q) == PGF_ERR_INVALID_ARG);
    pgf_params p;
    memset(&p, 0, sizeof(p));
    p.batch = 1; p.seqlen = 1; p.d_inner = 16; p.d_state = 16; p.n_dirs = 1;
    CHECK(pgf::make_plan(&p, nullptr) == PGF_ERR_INVALID_ARG);
    const int64_t big[] = {int64_t(1) << 40, INT64_MAX, -1, INT64_MIN};
    for (int64_t v : big) {
        pgf_params b = p;
        b.seqlen = v;
        CHECK(pgf::make_plan(&b, &q) != PGF_OK || v == (int64_t(1) << 40));
        b = p;
        b.d_inner = v;
        CHECK(pgf::make_plan(&b, &q) != PGF_OK);
        b = p;
        b.batch = v;
        CHECK(pgf::make_plan(&b, &q) != PGF_OK);
    }
    p.chunk_segs = 5000;
    CHECK(pgf::make_plan(&p, &q) == PGF_ERR_INVALID_ARG);
    // linear attention
    long la = 0;
    for (int64_t DK : {int64_t(8), int64_t(16), int64_t(32), int64_t(64)})
        for (int64_t DV : {int64_t(32), int64_t(64), int64_t(4096), int64_t(8192)})
            for (int64_t K : {int64_t(0), int64_t(1), int64_t(2), int64_t(3)})
                for (int seg : {0, -1, 64, 100}) {
                    pgf_la_params a;
                    memset(&a, 0, sizeof(a));
                    a.batch = 1; a.heads = 32; a.seqlen = 131072; a.d_key = DK; a.d_value = DV; a.n_dirs = K;
                    a.seg_len = seg;
                    pgf::LaPlan lq;
                    if (pgf::make_la_plan(&a, &lq) == PGF_OK) {
                        ++la;
                        CHECK(lq.state % 256 == 0 && lq.rec % 256 == 0 && lq.agg_h % 256 == 0 &&
                              lq.agg_s % 256 == 0 && lq.total % 256 == 0);
                        CHECK(lq.n_chunks * lq.chunk_len >= lq.L);
                    }
                }
    CHECK(pgf::make_la_plan(nullptr, nullptr) == PGF_ERR_INVALID_ARG);
    for (int s = -6; s <= 1; ++s) CHECK(strncmp(pgf_status_string(s), "PGF", 3) == 0);
    printf("plan driver: %ld plans checked, %ld argument sets rejected, %ld linear-attention plans, %d failures\n",
           plans, rejected, la, failures);
    return failures ? 1 : 0;
}
