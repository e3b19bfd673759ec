// libpgf entry points of the selective-SSM scans (include/pgf.h): argument
// checks, then the launch sequence of pgf_scan_kernels.h for the input type.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <mutex>

#include "pgf_plan.h"
#include "pgf_scan_launch.h"

// Workspace of pgf_scan_jvp_noalloc: a static device array, one per GPU the
// library runs on, alive until the process ends.  In host code `scratch` is
// a host-side stand-in, never a device address: the device address comes
// from hipGetSymbolAddress (scratch_address below).
static __device__ __align__(256) unsigned char scratch[PGF_SCRATCH_BYTES];

namespace pgf {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};

// The device address of this device's scratch array, looked up once per
// device (on the first call made with it current).  nullptr on failure.
void *scratch_address() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        (void)hipGetLastError();
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch[dev] = ptr;
    }
    return g_scratch[dev];
}

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
    return na && nb && pa < pb + nb && pb < pa + na;
}

// noalloc: the workspace is this device's static scratch array (p->workspace
// is not read), host blocks are sized to fit it, and the call creates no
// stream or event.
int scan_common(const void *x, const void *dx, const pgf_params *p, float *y, float *dy, float *d2y,
                void *stream, int order, bool noalloc = false) {
    Plan q;
    const int rc = make_plan(p, &q, noalloc ? (size_t)PGF_SCRATCH_BYTES : 0);
    if (rc != PGF_OK) return rc;
    if (q.order != order) return PGF_ERR_INVALID_ARG;
    if (!p->A || !p->b_delta || !p->W_B || !p->W_C) return PGF_ERR_INVALID_ARG;
    if (q.rank ? (!p->W_dx || !p->W_dt) : !p->w_delta) return PGF_ERR_INVALID_ARG;
    pgf_params pw = *p;
    if (noalloc) {
        if (q.ws.total > (size_t)PGF_SCRATCH_BYTES) return PGF_ERR_SCRATCH;
        q.noalloc = 1;
        pw.workspace = scratch_address();
        pw.workspace_bytes = PGF_SCRATCH_BYTES;
        if (!pw.workspace) return PGF_ERR_HIP;
    }
    p = &pw;
    if (!p->workspace || p->workspace_bytes < q.ws.total || ((uintptr_t)p->workspace & 255))
        return PGF_ERR_WORKSPACE;
    const size_t esz = q.in_bf16 ? 2 : 4;
    const size_t nx = (size_t)q.B * q.L * q.D;
    const size_t bx = nx * esz, bdx = nx * q.K * esz, by = nx * 4, bdy = nx * q.K * 4;
    if (q.L > 0) {
        if (!x || !dx || !y || !dy || (order == 2 && !d2y)) return PGF_ERR_INVALID_ARG;
        if (overlap(y, by, x, bx) || overlap(y, by, dx, bdx) || overlap(dy, bdy, x, bx) ||
            overlap(dy, bdy, dx, bdx) || overlap(y, by, dy, bdy))
            return PGF_ERR_INVALID_ARG;
        if (overlap(p->workspace, q.ws.total, y, by) || overlap(p->workspace, q.ws.total, dy, bdy) ||
            overlap(p->workspace, q.ws.total, x, bx) || overlap(p->workspace, q.ws.total, dx, bdx))
            return PGF_ERR_INVALID_ARG;
        if (order == 2 && (overlap(d2y, by, x, bx) || overlap(d2y, by, dx, bdx) || overlap(d2y, by, y, by) ||
                           overlap(d2y, by, dy, bdy) || overlap(d2y, by, p->workspace, q.ws.total)))
            return PGF_ERR_INVALID_ARG;
    }
    // Clear any stale error from earlier, unrelated work on this thread.
    (void)hipGetLastError();
    hipStream_t st = (hipStream_t)stream;
    if (q.in_bf16)
        return launch<uint16_t>(q, *p, (const uint16_t *)x, (const uint16_t *)dx, y, dy, d2y, st, nullptr, nullptr,
                                nullptr, nullptr);
    return launch<float>(q, *p, (const float *)x, (const float *)dx, y, dy, d2y, st, nullptr, nullptr, nullptr,
                         nullptr);
}

int param_common(const void *x, const float *gy, const pgf_params *p, float *y, float *gA, float *gB, float *gC,
                 void *stream) {
    Plan q;
    const int rc = make_plan(p, &q);
    if (rc != PGF_OK) return rc;
    if (q.order != 3) return PGF_ERR_INVALID_ARG;
    if (!p->A || !p->w_delta || !p->b_delta || !p->W_B || !p->W_C) return PGF_ERR_INVALID_ARG;
    if (!gA || !gB || !gC) return PGF_ERR_INVALID_ARG;
    // the residual weight's gradient, when there is a residual weight, and
    // the step size's, with its flows
    const float *gD = p->D_res ? p->grad_D_res : nullptr;
    if (p->D_res && !gD) return PGF_ERR_INVALID_ARG;
    const bool dlt = q.K == 4;
    if (dlt && (!p->grad_w_delta || !p->grad_b_delta)) return PGF_ERR_INVALID_ARG;
    if (!p->workspace || p->workspace_bytes < q.ws.total || ((uintptr_t)p->workspace & 255))
        return PGF_ERR_WORKSPACE;
    const size_t esz = q.in_bf16 ? 2 : 4;
    const size_t nx = (size_t)q.B * q.L * q.D;
    const size_t bx = nx * esz, bg = nx * 4, by = nx * 4, bw = q.ws.total;
    const float *grads[6] = {gA, gB, gC, gD, dlt ? p->grad_w_delta : nullptr, dlt ? p->grad_b_delta : nullptr};
    int ng = 3;
    for (int i = 3; i < 6; ++i)   // the per-channel gradients given, packed after the [D,N] ones
        if (grads[i]) grads[ng++] = grads[i];
    const size_t bnd = (size_t)q.N * q.D * 4, bd = (size_t)q.D * 4;
    const size_t bp[6] = {bnd, bnd, bnd, bd, bd, bd};
    for (int i = 0; i < ng; ++i) {
        for (int j = i + 1; j < ng; ++j)
            if (overlap(grads[i], bp[i], grads[j], bp[j])) return PGF_ERR_INVALID_ARG;
        if (overlap(grads[i], bp[i], p->workspace, bw)) return PGF_ERR_INVALID_ARG;
    }
    if (q.L > 0) {
        if (!x || !gy || !y) return PGF_ERR_INVALID_ARG;
        if (overlap(y, by, x, bx) || overlap(y, by, gy, bg) || overlap(y, by, p->workspace, bw) ||
            overlap(p->workspace, bw, x, bx) || overlap(p->workspace, bw, gy, bg))
            return PGF_ERR_INVALID_ARG;
        for (int i = 0; i < ng; ++i)
            if (overlap(grads[i], bp[i], x, bx) || overlap(grads[i], bp[i], gy, bg) ||
                overlap(grads[i], bp[i], y, by))
                return PGF_ERR_INVALID_ARG;
    }
    (void)hipGetLastError();
    hipStream_t st = (hipStream_t)stream;
    if (q.in_bf16)
        return launch<uint16_t>(q, *p, (const uint16_t *)x, nullptr, y, nullptr, nullptr, st, gy, gA, gB, gC);
    return launch<float>(q, *p, (const float *)x, nullptr, y, nullptr, nullptr, st, gy, gA, gB, gC);
}
}  // namespace
}  // namespace pgf

namespace pgf {
namespace {

// The plan, and whether the kernel tables cover it (host only).
int plan_checked(const pgf_params *p, pgf::Plan *q) {
    const int rc = pgf::make_plan(p, q);
    if (rc != PGF_OK) return rc;
    const bool ok = q->in_bf16 ? pgf::launch_supported<uint16_t>(*q, *p) : pgf::launch_supported<float>(*q, *p);
    return ok ? PGF_OK : PGF_ERR_UNSUPPORTED;
}

}  // namespace
}  // namespace pgf

extern "C" size_t pgf_workspace_bytes(const pgf_params *p) {
    pgf::Plan q;
    if (pgf::plan_checked(p, &q) != PGF_OK) return 0;
    return q.ws.total;
}

extern "C" int pgf_plan(const pgf_params *p, pgf_plan_info *info) {
    if (!info) return PGF_ERR_INVALID_ARG;
    pgf::Plan q;
    const int rc = pgf::plan_checked(p, &q);
    if (rc != PGF_OK) return rc;
    info->n_per_thread = q.nt;
    info->n_split = q.ns;
    info->seg_len = q.seg;
    info->chunk_segs = q.chunk_segs;
    info->chunk_len = q.chunk_len;
    info->n_chunks = q.n_chunks;
    info->workspace_bytes = q.ws.total;
    return PGF_OK;
}

extern "C" int pgf_param_grads(const void *x, const float *gy, const pgf_params *p, float *y, float *grad_A,
                               float *grad_B, float *grad_C, void *stream) {
    return pgf::param_common(x, gy, p, y, grad_A, grad_B, grad_C, stream);
}

extern "C" int pgf_scan_jvp(const void *x, const void *dx, const pgf_params *p, float *y, float *dy, void *stream) {
    return pgf::scan_common(x, dx, p, y, dy, nullptr, stream, 1);
}

extern "C" int pgf_scan_jvp_noalloc(const void *x, const void *dx, const pgf_params *p, float *y, float *dy,
                                    void *stream) {
    return pgf::scan_common(x, dx, p, y, dy, nullptr, stream, 1, true);
}

extern "C" int pgf_scan_jvp2(const void *x, const void *dx, const pgf_params *p, float *y, float *dy, float *d2y,
                             void *stream) {
    return pgf::scan_common(x, dx, p, y, dy, d2y, stream, 2);
}
