// A caller of libpgf through its C ABI alone (no Python, no torch): reads a
// problem from raw float32 files, runs pgf_scan_jvp on a stream of its own
// with a workspace it allocates, then pgf_scan_jvp_noalloc (no workspace) on
// the same stream, and writes both results back.  Used by
// tests/test_c_caller_gpu.py, which writes the inputs, compares the outputs
// with the fp64 oracle and the two calls with each other.
//
//   pgf_c_caller DIR
//   DIR/sizes.txt : B L D N K
//   DIR/{x,dx,A,w_delta,b_delta,W_B,W_C}.bin : row-major float32 arrays
//   writes DIR/y.bin [B,L,D], DIR/dy.bin [K,B,L,D] (pgf_scan_jvp) and
//   DIR/y_noalloc.bin, DIR/dy_noalloc.bin (pgf_scan_jvp_noalloc)
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "pgf.h"

namespace {

std::vector<float> read_f32(const std::string &path, size_t n) {
    std::vector<float> v(n);
    FILE *f = std::fopen(path.c_str(), "rb");
    if (!f || std::fread(v.data(), sizeof(float), n, f) != n) {
        std::fprintf(stderr, "cannot read %zu floats from %s\n", n, path.c_str());
        std::exit(2);
    }
    std::fclose(f);
    return v;
}

void write_f32(const std::string &path, const std::vector<float> &v) {
    FILE *f = std::fopen(path.c_str(), "wb");
    if (!f || std::fwrite(v.data(), sizeof(float), v.size(), f) != v.size()) {
        std::fprintf(stderr, "cannot write %s\n", path.c_str());
        std::exit(2);
    }
    std::fclose(f);
}

void hip_ok(hipError_t e, const char *what) {
    if (e != hipSuccess) {
        std::fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
        std::exit(3);
    }
}

float *to_device(const std::vector<float> &h) {
    void *d = nullptr;
    hip_ok(hipMalloc(&d, h.size() * sizeof(float) + 4), "hipMalloc");
    hip_ok(hipMemcpy(d, h.data(), h.size() * sizeof(float), hipMemcpyHostToDevice), "hipMemcpy H2D");
    return static_cast<float *>(d);
}

}  // namespace

int main(int argc, char **argv) {
    if (argc != 2) {
        std::fprintf(stderr, "usage: %s DIR\n", argv[0]);
        return 2;
    }
    const std::string dir = argv[1];
    long long B, L, D, N, K;
    FILE *fs = std::fopen((dir + "/sizes.txt").c_str(), "r");
    if (!fs || std::fscanf(fs, "%lld %lld %lld %lld %lld", &B, &L, &D, &N, &K) != 5) {
        std::fprintf(stderr, "cannot read sizes\n");
        return 2;
    }
    std::fclose(fs);
    const size_t nx = (size_t)(B * L * D);
    float *x = to_device(read_f32(dir + "/x.bin", nx));
    float *dx = to_device(read_f32(dir + "/dx.bin", nx * K));
    float *A = to_device(read_f32(dir + "/A.bin", (size_t)(D * N)));
    float *w = to_device(read_f32(dir + "/w_delta.bin", (size_t)D));
    float *b = to_device(read_f32(dir + "/b_delta.bin", (size_t)D));
    float *WB = to_device(read_f32(dir + "/W_B.bin", (size_t)(D * N)));
    float *WC = to_device(read_f32(dir + "/W_C.bin", (size_t)(D * N)));
    float *y = to_device(std::vector<float>(nx));
    float *dy = to_device(std::vector<float>(nx * K));

    pgf_params p = {};
    p.batch = B; p.seqlen = L; p.d_inner = D; p.d_state = N; p.n_dirs = K;
    p.in_dtype = PGF_F32;
    p.A = A; p.w_delta = w; p.b_delta = b; p.W_B = WB; p.W_C = WC;

    hipStream_t st;
    hip_ok(hipStreamCreate(&st), "hipStreamCreate");
    // without a workspace the call is refused before anything is launched
    int rc = pgf_scan_jvp(x, dx, &p, y, dy, st);
    std::printf("without workspace: %s\n", pgf_status_string(rc));
    if (rc != PGF_ERR_WORKSPACE) return 4;

    pgf_plan_info info;
    rc = pgf_plan(&p, &info);
    if (rc != PGF_OK) {
        std::printf("plan: %s\n", pgf_status_string(rc));
        return 4;
    }
    const size_t ws = pgf_workspace_bytes(&p);
    void *wsp = nullptr;
    hip_ok(hipMalloc(&wsp, ws), "hipMalloc workspace");
    p.workspace = wsp;
    p.workspace_bytes = ws;
    rc = pgf_scan_jvp(x, dx, &p, y, dy, st);
    std::printf("pgf_scan_jvp: %s (n_per_thread %d, n_split %d, seg_len %d, %lld host blocks, %zu workspace bytes)\n",
                pgf_status_string(rc), info.n_per_thread, info.n_split, info.seg_len, (long long)info.n_chunks, ws);
    if (rc != PGF_OK) return 4;
    hip_ok(hipStreamSynchronize(st), "hipStreamSynchronize");

    std::vector<float> hy(nx), hdy(nx * K);
    hip_ok(hipMemcpy(hy.data(), y, nx * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy D2H");
    hip_ok(hipMemcpy(hdy.data(), dy, nx * K * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy D2H");
    write_f32(dir + "/y.bin", hy);
    write_f32(dir + "/dy.bin", hdy);

    // the allocation-free entry point on the same stream, into cleared outputs
    hip_ok(hipMemsetAsync(y, 0, nx * sizeof(float), st), "hipMemsetAsync");
    hip_ok(hipMemsetAsync(dy, 0, nx * K * sizeof(float), st), "hipMemsetAsync");
    p.workspace = nullptr;
    p.workspace_bytes = 0;
    rc = pgf_scan_jvp_noalloc(x, dx, &p, y, dy, st);
    std::printf("pgf_scan_jvp_noalloc: %s\n", pgf_status_string(rc));
    if (rc != PGF_OK) return 4;
    hip_ok(hipStreamSynchronize(st), "hipStreamSynchronize");
    hip_ok(hipMemcpy(hy.data(), y, nx * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy D2H");
    hip_ok(hipMemcpy(hdy.data(), dy, nx * K * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy D2H");
    write_f32(dir + "/y_noalloc.bin", hy);
    write_f32(dir + "/dy_noalloc.bin", hdy);

    for (void *ptr : {(void *)x, (void *)dx, (void *)A, (void *)w, (void *)b, (void *)WB, (void *)WC, (void *)y,
                      (void *)dy, wsp})
        hip_ok(hipFree(ptr), "hipFree");
    hip_ok(hipStreamDestroy(st), "hipStreamDestroy");
    return 0;
}
