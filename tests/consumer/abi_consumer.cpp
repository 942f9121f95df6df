// A host program that uses the CPDP C ABI with nothing but the HIP runtime:
// its own device allocations, its own stream, no PyTorch.  It runs Algorithm 1
// (initialisation, then local steps and reconciles on the host cadence of
// cpdp_is_sync_step) on inputs read from files and writes the final state.
//
// usage: abi_consumer W P K steps T lr mu beta alpha param_dt dir [periods]
//   dir/theta0.bin        P parameters (fp32, or raw bf16 bits when param_dt = 1)
//   dir/grads_<s>.bin     W x P fp32 gradients of step s = 1..steps, replica-major
// writes dir/params.bin (W x P, parameter storage), dir/mom.bin (W x P fp32),
// dir/slow.bin and dir/anchor.bin (P fp32) and dir/kinds.txt (one line per step).
// Rows are padded to ld = P rounded up to 64 elements; the padding is filled
// with a byte pattern before the run and checked untouched afterwards.
// With a trailing `periods` argument it then times that many further periods
// on the last gradients and prints the host time per C-ABI call (validation
// and enqueue, no synchronisation) and the device time per period.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "cpdp.h"

#define HIP_OK(x)                                                                   \
    do {                                                                            \
        hipError_t e_ = (x);                                                        \
        if (e_ != hipSuccess) {                                                     \
            std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));     \
            return 1;                                                               \
        }                                                                           \
    } while (0)

#define CPDP_OK_(x)                                                                 \
    do {                                                                            \
        int s_ = (x);                                                               \
        if (s_ != CPDP_OK) {                                                        \
            std::fprintf(stderr, "%s failed: %s\n", #x, cpdp_status_str(s_));       \
            return 1;                                                               \
        }                                                                           \
    } while (0)

static bool read_file(const std::string& path, void* dst, size_t bytes) {
    FILE* f = std::fopen(path.c_str(), "rb");
    if (!f) return false;
    const bool ok = std::fread(dst, 1, bytes, f) == bytes;
    std::fclose(f);
    return ok;
}

static bool write_file(const std::string& path, const void* src, size_t bytes) {
    FILE* f = std::fopen(path.c_str(), "wb");
    if (!f) return false;
    const bool ok = std::fwrite(src, 1, bytes, f) == bytes;
    std::fclose(f);
    return ok;
}

static constexpr unsigned char kPad = 0x5A;

int main(int argc, char** argv) {
    if (argc != 12 && argc != 13) {
        std::fprintf(stderr, "usage: %s W P K steps T lr mu beta alpha param_dt dir [periods]\n",
                     argv[0]);
        return 2;
    }
    const int time_periods = argc == 13 ? std::atoi(argv[12]) : 0;
    const int W = std::atoi(argv[1]);
    const int64_t P = std::atoll(argv[2]);
    const int K = std::atoi(argv[3]);
    const int steps = std::atoi(argv[4]);
    const int64_t T = std::atoll(argv[5]);
    const float lr = std::strtof(argv[6], nullptr), mu = std::strtof(argv[7], nullptr);
    const float beta = std::strtof(argv[8], nullptr), alpha = std::strtof(argv[9], nullptr);
    const int pdt = std::atoi(argv[10]);
    const std::string dir = argv[11];
    if (W < 1 || P < 1 || K < 1 || steps < 1 || T < 0 || (pdt != CPDP_F32 && pdt != CPDP_BF16)) {
        std::fprintf(stderr, "bad arguments\n");
        return 2;
    }
    const size_t ps = pdt == CPDP_BF16 ? 2 : 4;
    const int64_t ld = (P + 63) / 64 * 64;

    std::vector<unsigned char> theta0(P * ps);
    if (!read_file(dir + "/theta0.bin", theta0.data(), theta0.size())) {
        std::fprintf(stderr, "cannot read theta0.bin\n");
        return 1;
    }

    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    void *d_theta0, *d_params, *d_mom, *d_grads;
    float *d_slow, *d_anchor;
    HIP_OK(hipMalloc(&d_theta0, P * ps));
    HIP_OK(hipMalloc(&d_params, W * ld * ps));
    HIP_OK(hipMalloc(&d_mom, W * ld * 4));
    HIP_OK(hipMalloc(&d_grads, W * ld * 4));
    HIP_OK(hipMalloc(&d_slow, P * 4));
    HIP_OK(hipMalloc(&d_anchor, P * 4));
    HIP_OK(hipMemset(d_params, kPad, W * ld * ps));
    HIP_OK(hipMemset(d_mom, kPad, W * ld * 4));
    HIP_OK(hipMemcpy(d_theta0, theta0.data(), P * ps, hipMemcpyHostToDevice));

    CPDP_OK_(cpdp_state_init(d_theta0, d_params, d_mom, d_slow, d_anchor, W, P, ld, K, pdt,
                             CPDP_F32, stream));
    std::vector<float> g(W * P);
    std::string kinds;
    for (int s = 1; s <= steps; ++s) {
        if (!read_file(dir + "/grads_" + std::to_string(s) + ".bin", g.data(), g.size() * 4)) {
            std::fprintf(stderr, "cannot read grads_%d.bin\n", s);
            return 1;
        }
        // the host buffer is reused next step: wait for the copy before refilling it
        HIP_OK(hipMemcpy2DAsync(d_grads, ld * 4, g.data(), P * 4, P * 4, W,
                                hipMemcpyHostToDevice, stream));
        const int64_t t = T > 0 ? (s - 1) % T + 1 : s;
        const int sync = cpdp_is_sync_step(t, K, T);
        if (sync < 0) {
            std::fprintf(stderr, "cpdp_is_sync_step: %s\n", cpdp_status_str(-sync));
            return 1;
        }
        if (sync)
            CPDP_OK_(cpdp_reconcile(d_params, d_mom, d_grads, d_slow, d_anchor, W, P, ld, K, lr,
                                    mu, beta, alpha, pdt, CPDP_F32, CPDP_F32, stream));
        else
            CPDP_OK_(cpdp_local_step(d_params, d_mom, d_grads, W, P, ld, K, lr, mu, pdt,
                                     CPDP_F32, CPDP_F32, stream));
        HIP_OK(hipStreamSynchronize(stream));
        kinds += sync ? "reconcile\n" : "local\n";
    }

    if (time_periods > 0) {
        hipEvent_t e0, e1;
        HIP_OK(hipEventCreate(&e0));
        HIP_OK(hipEventCreate(&e1));
        double host_s = 0.0;
        int64_t calls = 0;
        HIP_OK(hipEventRecord(e0, stream));
        for (int r = 0; r < time_periods; ++r) {
            for (int t = 1; t <= K; ++t) {
                const auto h0 = std::chrono::steady_clock::now();
                const int sync = cpdp_is_sync_step(t, K, 0);
                const int st = sync ? cpdp_reconcile(d_params, d_mom, d_grads, d_slow, d_anchor, W,
                                                     P, ld, K, lr, mu, beta, alpha, pdt, CPDP_F32,
                                                     CPDP_F32, stream)
                                    : cpdp_local_step(d_params, d_mom, d_grads, W, P, ld, K, lr,
                                                      mu, pdt, CPDP_F32, CPDP_F32, stream);
                host_s += std::chrono::duration<double>(std::chrono::steady_clock::now() - h0).count();
                ++calls;
                if (st != CPDP_OK) {
                    std::fprintf(stderr, "timed call failed: %s\n", cpdp_status_str(st));
                    return 1;
                }
            }
        }
        HIP_OK(hipEventRecord(e1, stream));
        HIP_OK(hipEventSynchronize(e1));
        float ms = 0.0f;
        HIP_OK(hipEventElapsedTime(&ms, e0, e1));
        std::printf("timing: %d periods of K=%d, host %.2f us per call (cadence, validation, "
                    "enqueue), device %.2f us per period\n",
                    time_periods, K, 1e6 * host_s / (double)calls, 1e3 * ms / time_periods);
        HIP_OK(hipEventDestroy(e0));
        HIP_OK(hipEventDestroy(e1));
    }

    std::vector<unsigned char> params(W * ld * ps);
    std::vector<unsigned char> mom(W * ld * 4);
    std::vector<float> slow(P), anchor(P);
    HIP_OK(hipMemcpy(params.data(), d_params, params.size(), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(mom.data(), d_mom, mom.size(), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(slow.data(), d_slow, P * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(anchor.data(), d_anchor, P * 4, hipMemcpyDeviceToHost));

    // the padding columns [P, ld) of every row must be untouched
    for (int i = 0; i < W; ++i) {
        for (int64_t b = P * (int64_t)ps; b < ld * (int64_t)ps; ++b)
            if (params[i * ld * ps + b] != kPad) { std::fprintf(stderr, "params pad written\n"); return 1; }
        for (int64_t b = P * 4; b < ld * 4; ++b)
            if (mom[i * ld * 4 + b] != kPad) { std::fprintf(stderr, "mom pad written\n"); return 1; }
    }
    std::vector<unsigned char> pp(W * P * ps), mm(W * P * 4);
    for (int i = 0; i < W; ++i) {
        std::memcpy(&pp[i * P * ps], &params[i * ld * ps], P * ps);
        std::memcpy(&mm[i * P * 4], &mom[i * ld * 4], P * 4);
    }
    if (!write_file(dir + "/params.bin", pp.data(), pp.size()) ||
        !write_file(dir + "/mom.bin", mm.data(), mm.size()) ||
        !write_file(dir + "/slow.bin", slow.data(), P * 4) ||
        !write_file(dir + "/anchor.bin", anchor.data(), P * 4) ||
        !write_file(dir + "/kinds.txt", kinds.data(), kinds.size())) {
        std::fprintf(stderr, "cannot write outputs\n");
        return 1;
    }
    HIP_OK(hipFree(d_theta0));
    HIP_OK(hipFree(d_params));
    HIP_OK(hipFree(d_mom));
    HIP_OK(hipFree(d_grads));
    HIP_OK(hipFree(d_slow));
    HIP_OK(hipFree(d_anchor));
    HIP_OK(hipStreamDestroy(stream));
    std::printf("ok %d steps\n", steps);
    return 0;
}
