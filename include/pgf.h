/*
 * pgf.h -- C ABI of libpgf: the fused primal + tangent (forward-mode JVP)
 * scan of a selective diagonal state-space model on AMD Instinct MI355X
 * (gfx950).
 *
 * The operation (paper Sec. 3, Lemma 3.1 "Selectivity Jacobian", Eq. 3;
 * Prop. 3.2, Eq. 4; Alg. 1 "Tiled Operator-Space Evolution"):
 *
 *   For every batch b, channel d, state n and step t = 0 .. L-1
 *     z      = x[b,t,d] * w_delta[d] + b_delta[d]
 *     Delta  = softplus(z)                      selective step size
 *     Abar   = exp(Delta * A[d,n])              zero-order-hold transition
 *     B_t[n] = sum_d' x[b,t,d'] W_B[d',n] + b_B[n]
 *     C_t[n] = sum_d' x[b,t,d'] W_C[d',n] + b_C[n]
 *     h      = Abar * h + Delta * B_t[n] * x[b,t,d]        primal state
 *     y[b,t,d] = sum_n C_t[n] * h                          output map
 *   and, for every tangent direction k (the input perturbation dx_k), the
 *   exact directional derivative of all of the above along dx_k:
 *     dDelta = sigmoid(z) * w_delta[d] * dx_k[b,t,d]
 *     dB[n], dC[n] = the projections applied to dx_k (no bias)
 *     dh     = Abar*dh + Abar*A[d,n]*dDelta*h_prev
 *              + dDelta*B*x + Delta*dB*x + Delta*B*dx      (Eq. 3: K_t, j_t)
 *     dy_k[b,t,d] = sum_n dC[n]*h + C[n]*dh
 *   The state starts at h_in / dh_in (zero when NULL).  The dC*h term is the
 *   derivative of the output map through C; the paper's output variation
 *   (Eq. 2) leaves it out, this library differentiates the map in full.
 *
 * Only the O(B*D*N*(1+K)) state crosses from one block of steps to the next
 * (the block hand-off of Alg. 1); the state trajectory is never stored, so
 * the workspace does not depend on L (Sec. 4.3, memory theorem).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers (x, dx, y, dy, parameters, h_in/dh_in/h_out/dh_out,
 *     workspace) are DEVICE pointers owned by the caller.  The library
 *     never allocates or frees device memory.
 *   - Layouts are dense row-major, last index fastest:
 *       x [B,L,D]     dx [K,B,L,D]     y [B,L,D] (f32)   dy [K,B,L,D] (f32)
 *       A, W_B, W_C [D,N]   w_delta, b_delta [D]   b_B, b_C [N]
 *       h_in, h_out [B,D,N]   dh_in, dh_out [K,B,D,N]            (all f32)
 *   - x and dx are f32 or bf16 (in_dtype); everything else is f32, and all
 *     arithmetic of the scan runs in f32.
 *   - Calls are asynchronous on `stream` and make no host<->device sync.
 *     Argument checks are synchronous and happen before any launch; on a
 *     failed check nothing is launched and the outputs are untouched.
 *     Faults inside kernels surface at the caller's next synchronisation.
 *   - A call whose sequence spans several host blocks runs the projections
 *     of the next block on a helper stream of the device (default priority,
 *     created on first use and kept until the process ends), forked from
 *     and joined back to `stream` with events: the call stays ordered with
 *     the work on `stream` before and after it, also under stream capture.
 *   - Launches go to the device that is current on the calling thread; the
 *     stream must belong to it.
 *   - Apart from the helper streams and the optional launch-timing record
 *     (see pgf_timing_*) the library keeps no state between calls.  It is
 *     reentrant on distinct workspaces (calls from several host threads
 *     that use one device's helper enqueue one at a time).  Two calls in
 *     flight on the same workspace race.
 *   - No C++ exception crosses this boundary.
 */
#ifndef PGF_H_
#define PGF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (negative = error). */
#define PGF_OK                 0
#define PGF_ERR_INVALID_ARG   -1   /* NULL where a pointer is required, bad size, overlap  */
#define PGF_ERR_UNSUPPORTED   -2   /* shape outside what the kernels are built for          */
#define PGF_ERR_WORKSPACE     -3   /* workspace NULL or smaller than pgf_workspace_bytes    */
#define PGF_ERR_HIP           -4   /* a HIP launch or runtime call failed                   */
#define PGF_ERR_SCRATCH       -5   /* pgf_scan_jvp_noalloc: the call needs more than
                                      PGF_SCRATCH_BYTES of workspace                       */

/* dtype of x and dx. */
#define PGF_F32   0
#define PGF_BF16  1

/* Input drive of the discretised recurrence (pgf_params.drive). */
#define PGF_DRIVE_EULER  0   /* b = Delta * B * x                                  */
#define PGF_DRIVE_ZOH    1   /* b = A^-1 (Abar - 1) * B * x (zero-order hold)      */

/* Output activation (pgf_params.activation). */
#define PGF_ACT_IDENTITY 0
#define PGF_ACT_SILU     1   /* act(v) = v * sigmoid(v)                            */

typedef struct pgf_params {
    /* Problem size: batch B, sequence length L (>= 0), channels D, state size
     * N, tangent directions K.  Supported: B, D >= 1; N in {4,8,16,32,64};
     * 1 <= K <= 8. */
    int64_t batch, seqlen, d_inner, d_state, n_dirs;
    int32_t in_dtype;      /* PGF_F32 or PGF_BF16                                       */
    /* Tiling overrides, 0 = library default (the defaults depend on B, D, N,
     * K and in_dtype only, never on L).
     *   seg_len   : steps per segment of the parallel-in-L evaluation (a
     *               power of two, 16 .. 65536), or -1 to force the
     *               sequential-in-L evaluation.
     *   chunk_segs: segments per host block (the Alg. 1 block is
     *               chunk_segs*seg_len steps), 1 .. 4096.
     * Results are bit-identical for every chunk_segs at a fixed seg_len. */
    int32_t seg_len;
    int32_t chunk_segs;
    /* Which flows a call carries; read by the planning calls too.
     *   0 or 1: first order (pgf_scan_jvp).
     *   2: second order (pgf_scan_jvp2; needs n_dirs == 2; any N).
     *   3: parameter flows (pgf_param_grads; any N; n_dirs is not read). */
    int32_t order;
    /* Model parameters (device, f32).  b_B / b_C may be NULL (= 0). */
    const float *A, *w_delta, *b_delta, *W_B, *W_C, *b_B, *b_C;
    /* Optional state hand-off (device, f32; NULL = zero in / not written).
     * Passing one call's h_out/dh_out as the next call's h_in/dh_in over the
     * continuation of the sequence reproduces one long call bit for bit when
     * the first call's L is a multiple of the segment length. */
    const float *h_in, *dh_in;
    float *h_out, *dh_out;
    /* Scratch (device), at least pgf_workspace_bytes(p) bytes, 256-byte
     * aligned.  Its size does not depend on L. */
    void *workspace;
    size_t workspace_bytes;
    /* Second order only: state of the mixed flow, [B,D,N] (NULL = zero in /
     * not written). */
    const float *d2h_in;
    float *d2h_out;
    /* Model variants of the first-order scan and of the parameter flows
     * (Sec. 3 output map, the appendix's zero-order-hold drive); zero for
     * the second order.  With any of them set, pgf_scan_jvp supports
     * N <= 16 and K <= 2 for a real A (every N and K for a complex A;
     * pgf_param_grads: every N).
     *   drive      : PGF_DRIVE_EULER or PGF_DRIVE_ZOH
     *   activation : PGF_ACT_IDENTITY or PGF_ACT_SILU
     *   D_res      : device, [D] f32 residual weight, or NULL (= 0)
     * The output becomes y = act(sum_n C h + D_res x) and
     * dy_k = act'(.) * (sum_n dC_k h + C dh_k + D_res dx_k). */
    int32_t drive;
    int32_t activation;
    const float *D_res;
    /* Complex diagonal transition (Sec. 3, state in C^{D x N}): the
     * imaginary part of A, device [D,N] f32, or NULL for a real A.  With it
     * the output is y = sum_n C Re(h) and dy_k = sum_n dC_k Re(h) + C Re(dh_k),
     * and with the output map above y = act(sum_n C Re(h) + D_res x) (Sec.
     * 3's general form); h_in/h_out are [B,D,N] and dh_in/dh_out [K,B,D,N]
     * complex (interleaved real, imaginary f32).  Either drive: with the
     * zero-order hold the drive coefficient is the complex (Abar - 1) / A.
     * First order only (every N and K of it). */
    const float *A_im;
    /* Channel groups with their own B and C (Mamba-style grouped
     * projections), 0 or 1 = one group.  With G > 1 groups, W_B and W_C are
     * [D, G*N], b_B and b_C [G*N], and channel d uses the columns
     * [gN, (g+1)N) of group g = d / (D/G).  D/G must be a multiple of 64
     * and G*N a power of two, at most 64.  First order only, Euler drive (the output map is
     * allowed), N <= 16, K <= 2. */
    int32_t n_groups;
    /* Low-rank step size (the Mamba step-size projection through a rank-R
     * bottleneck over all channels, Sec. 3 with z_t = W_dt (W_dx^T x_t) + b):
     * dt_rank = R in 1..128, or 0 for the per-channel step size above.  With
     * R > 0 the step size is Delta = softplus(z), z = (x W_dx) W_dt +
     * b_delta, and its tangent dDelta_k = sigmoid(z) (dx_k W_dx) W_dt;
     *   W_dx : device, [D, R] f32, row-major
     *   W_dt : device, [R, D] f32, row-major
     * w_delta is not read (may be NULL).  First order only, Euler drive (the
     * output map is allowed), one group, real A, N <= 16, K <= 2.  The
     * workspace then also holds z and dz_k of one host block, [1+K][B][Tc][D]
     * f32, and may reach 2 GiB. */
    int32_t dt_rank;
    const float *W_dx, *W_dt;
    /* Parameter flows with D_res set: dl/dD_res, device [D] f32, ADDED to
     * (like grad_A); not read otherwise. */
    float *grad_D_res;
    /* Parameter flows only (read by the planning calls too): 1 to also carry
     * the flows of the step size's parameters w_delta and b_delta (see
     * pgf_param_grads), 0 not to.  With it, grad_w_delta and grad_b_delta
     * (device, [D] f32, ADDED to) receive dl/dw_delta and dl/db_delta, and
     * dh_in/dh_out hold four planes. */
    int32_t delta_flows;
    float *grad_w_delta, *grad_b_delta;
} pgf_params;

/* How a call is tiled (host-side planning; no device access). */
typedef struct pgf_plan_info {
    int32_t n_per_thread;   /* states n held by one thread                          */
    int32_t n_split;        /* threads sharing one channel (N / n_per_thread)       */
    int32_t seg_len;        /* segment length, or 0 in the sequential evaluation    */
    int32_t chunk_segs;     /* segments per host block                              */
    int64_t chunk_len;      /* steps per host block                                 */
    int64_t n_chunks;       /* host blocks for this L                               */
    size_t  workspace_bytes;
} pgf_plan_info;

/* Bytes of workspace a call with these sizes needs.  Reads the size
 * fields, in_dtype, seg_len, chunk_segs, order, drive, activation,
 * n_groups and dt_rank, and tests D_res and A_im for NULL (never
 * dereferenced).  Returns 0 if the sizes are invalid or unsupported.  Host
 * only. */
size_t pgf_workspace_bytes(const pgf_params *p);

/* Fill *info with the tiling a call would use.  Host only.  Returns a status. */
int pgf_plan(const pgf_params *p, pgf_plan_info *info);

/* The fused primal + tangent scan (see the file comment).
 *   x  : device, [B,L,D] in in_dtype            (read)
 *   dx : device, [K,B,L,D] in in_dtype          (read)
 *   y  : device, [B,L,D] f32                    (fully overwritten)
 *   dy : device, [K,B,L,D] f32                  (fully overwritten)
 *   stream : a hipStream_t (NULL = the default stream)
 * y and dy must not overlap x, dx or each other, and the workspace none of
 * them.  Returns PGF_OK or an error code; see the conventions above. */
int pgf_scan_jvp(const void *x, const void *dx, const pgf_params *p,
                 float *y, float *dy, void *stream);

/* For callers that cannot allocate device memory or create streams (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): pgf_scan_jvp with its workspace taken from a static device
 * array of the library, PGF_SCRATCH_BYTES per GPU it runs on, held until
 * the process ends.  Arguments and outputs as pgf_scan_jvp, except:
 *   - p->workspace and p->workspace_bytes are not read;
 *   - with chunk_segs = 0 the host blocks are sized so that the workspace
 *     fits the scratch array; a call that cannot fit it (its state alone,
 *     or an explicit chunk_segs too large) returns PGF_ERR_SCRATCH before
 *     anything is launched;
 *   - every host block runs in order on `stream` (no helper stream), and
 *     the call records no timing events;
 *   - the first call on a device looks up that device's array
 *     (hipGetSymbolAddress); no call allocates, frees or creates anything.
 * Outputs equal pgf_scan_jvp's bit for bit (results do not depend on the
 * host-block size).  Every call on one GPU uses the same array, which keeps
 * the last call's contents (each call writes every part of it before
 * reading it): calls that overlap in time on one GPU race, from any stream
 * or thread. */
#define PGF_SCRATCH_BYTES ((size_t)256 << 20)
int pgf_scan_jvp_noalloc(const void *x, const void *dx, const pgf_params *p,
                         float *y, float *dy, void *stream);

/* Second-order flow (App. G, the Hessian flow): along the two input
 * directions v = dx[0] and w = dx[1], the primal, both first-order flows and
 * the mixed second directional derivative, with the curvature of
 * Delta = softplus(z) (softplus'' = sigmoid*(1-sigmoid)) and the
 * cross-talk terms of the transition:
 *   h_vw = Abar*h_vw + Abar_w*h_v + Abar_v*h_w + Abar_vw*h + b_vw,
 *   Abar_vw = Abar*A^2*dDelta_v*dDelta_w + Abar*A*d2Delta_vw,
 *   d2y[b,t,d] = sum_n dC_v h_w + dC_w h_v + C h_vw.
 *   x   : device, [B,L,D] in in_dtype      dx : device, [2,B,L,D] (v, w)
 *   y   : device, [B,L,D] f32              dy : device, [2,B,L,D] f32
 *   d2y : device, [B,L,D] f32 (the mixed flow's output)
 * p->order must be 2 and p->n_dirs 2; h_in/dh_in/h_out/dh_out and
 * d2h_in/d2h_out carry the state as in pgf_scan_jvp.  y and dy equal what
 * pgf_scan_jvp returns for the same two directions up to rounding.  Other
 * conventions as pgf_scan_jvp; d2y must not overlap any other array. */
int pgf_scan_jvp2(const void *x, const void *dx, const pgf_params *p,
                  float *y, float *dy, float *d2y, void *stream);

/* Parameter-sensitivity flows with online gradient accumulation (App. E,
 * Alg. 2 "online parameter gradient accumulation").  Given the adjoint
 * signal gy = dl/dy of a scalar loss l, runs the primal scan and, in the
 * same pass, the flows of the state's sensitivity to the parameters, per
 * lane (b, d, n):
 *   GammaA' = Abar*GammaA + Delta*Abar*h       (dh/dA[d,n]; the Euler drive
 *                                              Delta*B*x has no A in it)
 *   GammaB' = Abar*GammaB + Delta*x            (dh/dB for a per-lane offset)
 *   h'      = Abar*h + Delta*B_t[n]*x,  y = sum_n C_t[n]*h'
 * and accumulates, over b and t,
 *   grad_A[d,n] += gy*C_t[n]*GammaA'     = dl/dA
 *   grad_B[d,n] += gy*C_t[n]*GammaB'     = dl/d(offset of B_t[n] in lane d,n)
 *   grad_C[d,n] += gy*h'                 = dl/d(offset of C_t[n] in lane d,n)
 * (the outer product of the adjoint and the state).  Summing grad_B and
 * grad_C over d gives dl/db_B and dl/db_C.  No trajectory is stored.
 *   x      : device, [B,L,D] in in_dtype            (read)
 *   gy     : device, [B,L,D] f32, the adjoint signal (read)
 *   y      : device, [B,L,D] f32                    (fully overwritten)
 *   grad_A, grad_B, grad_C : device, [D,N] f32, ADDED to (the caller zeroes
 *            them before the first call of a sequence)
 *   stream : a hipStream_t (NULL = the default stream)
 * Output map (Sec. 3; p->activation, p->D_res as in pgf_scan_jvp): with
 * y = act(yhat), yhat = sum_n C_t[n]*h' + D_res*x, the adjoint reaches the
 * state through w = gy*act'(yhat) (the sigma' factor of Alg. 2's G_C
 * update), so gy is replaced by w in the three sums above, and
 *   p->grad_D_res[d] += w*x              = dl/dD_res
 * (grad_D_res is required when D_res is set).  The ZOH drive
 * (p->drive) adds (de/dA)*B_t[n]*x to GammaA' with e = (Abar - 1)/A, and
 * takes e in place of Delta in the other drives.
 * Step-size parameters (p->delta_flows = 1; Sec. 3, Delta = softplus(z),
 * z = w_delta*x + b_delta, sigma = sigmoid(z) = dDelta/db_delta and
 * sigma*x = dDelta/dw_delta): the state moves with Delta by
 *   hd = A*Abar*h + Abar^z*B_t[n]*x  (z = 1 with ZOH, 0 with Euler),
 * so two more flows per lane run beside the others,
 *   Gamma_w' = Abar*Gamma_w + sigma*x*hd,  Gamma_s' = Abar*Gamma_s + sigma*hd,
 * and per channel
 *   grad_w_delta[d] += w*sum_n C_t[n]*Gamma_w',
 *   grad_b_delta[d] += w*sum_n C_t[n]*Gamma_s'
 * (w = gy*act'(yhat), or gy).  dh_in/dh_out then hold
 * [GammaA; GammaB; Gamma_w; Gamma_s] as [4,B,D,N].
 * p->order must be 3.  State hand-off: h_in/h_out as in pgf_scan_jvp;
 * dh_in/dh_out hold [GammaA; GammaB] as [2,B,D,N] (four planes with
 * delta_flows).  Chaining calls through
 * the state and adding into the same gradients gives the gradients of the
 * whole sequence (up to the rounding of the additions).  y must not overlap
 * x or gy; the gradients must not overlap any other array or each other;
 * the workspace must not overlap x, gy, y or the gradients.  Other
 * conventions as pgf_scan_jvp. */
int pgf_param_grads(const void *x, const float *gy, const pgf_params *p,
                    float *y, float *grad_A, float *grad_B, float *grad_C, void *stream);

/* ------------------------------------------------------------------------
 * Decaying linear attention with its tangent flow (App. F: linear
 * transformers, RetNet, RWKV-6 as general linear recurrences).  Per batch b
 * and head h the state is a d_key x d_value matrix S with a per-key-dimension
 * decay alpha_t = exp(g_t), g_t the log-decay (an input; g <= 0 decays):
 *   S_t[i,j] = alpha_t[i]*S_{t-1}[i,j] + k_t[i]*v_t[j],  o_t[j] = sum_i q_t[i]*S_t[i,j]
 * and, for each of K tangent directions (dq, dk, dv, dg) of the four input
 * sequences, the total differential (d alpha = alpha*dg):
 *   dS_t = alpha*dS_{t-1} + (alpha*dg)*S_{t-1} + dk*v^T + k*dv^T
 *   do_t = S_t^T dq + dS_t^T q
 * RetNet is a constant scalar decay, a linear transformer without
 * normaliser g = 0.  As for the SSM, only the O(B*H*dk*dv*(1+K)) state
 * crosses from one block of steps to the next and the workspace does not
 * depend on L.
 * ------------------------------------------------------------------------ */
typedef struct pgf_la_params {
    /* Sizes.  Supported: d_key in {16, 32, 64}; d_value a multiple of 64
     * (at most 4096); n_dirs in {1, 2}; batch, heads >= 1; seqlen >= 0. */
    int64_t batch, heads, seqlen, d_key, d_value, n_dirs;
    /* Tiling overrides as in pgf_params (0 = default, seg_len -1 =
     * sequential in L); results are bit-identical for every chunk_segs at
     * a fixed seg_len. */
    int32_t seg_len, chunk_segs;
    /* Optional state hand-off (device, f32; NULL = zero in / not written):
     * S [B,H,dk,dv], dS [K,B,H,dk,dv]. */
    const float *S_in, *dS_in;
    float *S_out, *dS_out;
    /* Scratch (device), at least pgf_la_workspace_bytes(p), 256-byte aligned. */
    void *workspace;
    size_t workspace_bytes;
} pgf_la_params;

/* Workspace bytes for these sizes (0 if invalid or unsupported).  Host only. */
size_t pgf_la_workspace_bytes(const pgf_la_params *p);

/* Tiling of a call (n_per_thread = d_key, n_split = 1).  Host only. */
int pgf_la_plan(const pgf_la_params *p, pgf_plan_info *info);

/* The primal and tangent scan.  All arrays device, f32, dense row-major:
 *   q, k, g      [B,H,L,dk]        v   [B,H,L,dv]                 (read)
 *   dq, dk, dg   [K,B,H,L,dk]      dv  [K,B,H,L,dv]               (read)
 *   o            [B,H,L,dv]        do_ [K,B,H,L,dv]   (fully overwritten)
 * o and do_ must not overlap any input or each other, and the workspace
 * none of them.  Conventions as pgf_scan_jvp (asynchronous on stream,
 * checks before any launch, current device). */
int pgf_la_scan_jvp(const float *q, const float *k, const float *v, const float *g,
                    const float *dq, const float *dk, const float *dv, const float *dg,
                    const pgf_la_params *p, float *o, float *do_, void *stream);

/* Static string for a status code. */
const char *pgf_status_string(int status);

/* Launch timing (measurement aid, off by default).  While enabled, every
 * kernel a call launches is bracketed by HIP events on the call's stream;
 * pgf_timing_read synchronises those events and returns, per kernel kind
 * (0 projection, 1 segment aggregate, 2 carry, 3 scan+outputs, 4 state
 * import/export), the summed milliseconds and launch counts, then clears
 * the record.  Arrays have PGF_TIMING_KINDS entries.  Not reentrant. */
#define PGF_TIMING_KINDS 5
int pgf_timing_enable(int on);
int pgf_timing_read(double *ms, int64_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* PGF_H_ */
