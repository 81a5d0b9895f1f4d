// A native consumer of the C ABI: device buffers from hipMalloc, a HIP
// stream of its own, libiabn's training forward and backward called through
// include/iabn.h (no Python, no torch), checked against the oracle's C
// library on the same inputs.  Test infrastructure (it links the oracle).
//
// usage: iabn_abi_check N C HW dtype(0 f32, 1 f16, 2 bf16) seed
// exit status 0 when every output is within the parity gate.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "iabn.h"

extern "C" {
void oracle_forward_train(const double* x, int64_t N, int64_t C, int64_t HW, const double* gamma,
                          const double* beta, double eps, double momentum, double slope,
                          double* running_mean, double* running_var, double* z, double* mean,
                          double* var);
void oracle_backward_i(const double* z, const double* dz, int64_t N, int64_t C, int64_t HW,
                       const double* gamma, const double* beta, const double* var, double eps,
                       double slope, double* dx, double* dgamma, double* dbeta);
}

#define CHECK_HIP(x)                                                                   \
    do {                                                                               \
        hipError_t e_ = (x);                                                           \
        if (e_ != hipSuccess) {                                                        \
            fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            exit(2);                                                                   \
        }                                                                              \
    } while (0)

#define CHECK_IABN(x)                                                                  \
    do {                                                                               \
        int s_ = (x);                                                                  \
        if (s_ != IABN_OK) {                                                           \
            fprintf(stderr, "libiabn: %s (%s) at line %d\n", iabn_status_string(s_),   \
                    iabn_last_error(), __LINE__);                                      \
            exit(2);                                                                   \
        }                                                                              \
    } while (0)

// Seeded inputs: a 64-bit LCG and Box-Muller, per-channel mean and spread.
struct Rng {
    uint64_t s;
    double uniform() {
        s = s * 6364136223846793005ull + 1442695040888963407ull;
        return ((s >> 11) + 0.5) * (1.0 / 9007199254740992.0);
    }
    double normal() {
        const double u = uniform(), v = uniform();
        return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
    }
};

// Rounds to the storage type (nearest even) and returns the stored bits
// and their exact value.  bf16 rounds through float32, as the library's
// conversions do.
static double bf16_bits_to_double(uint16_t b) {
    const uint32_t u = static_cast<uint32_t>(b) << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static uint32_t store(double v, int dtype, double* exact) {
    if (dtype == IABN_F32) {
        const float f = static_cast<float>(v);
        *exact = f;
        uint32_t b;
        memcpy(&b, &f, 4);
        return b;
    }
    if (dtype == IABN_F16) {
        const _Float16 h = static_cast<_Float16>(v);
        *exact = static_cast<double>(h);
        uint16_t b;
        memcpy(&b, &h, 2);
        return b;
    }
    const float f = static_cast<float>(v);
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    const uint16_t b = static_cast<uint16_t>(u >> 16);
    *exact = bf16_bits_to_double(b);
    return b;
}

static double load(const std::vector<uint8_t>& buf, size_t i, int dtype) {
    if (dtype == IABN_F32) {
        float f;
        memcpy(&f, &buf[4 * i], 4);
        return f;
    }
    uint16_t b;
    memcpy(&b, &buf[2 * i], 2);
    if (dtype == IABN_F16) {
        _Float16 h;
        memcpy(&h, &b, 2);
        return static_cast<double>(h);
    }
    return bf16_bits_to_double(b);
}

// max_i |g_i - r_i| / max(|r_i|, 1e-3 max_j |r_j|)
static double max_rel(const std::vector<double>& g, const std::vector<double>& r) {
    double mx = 0.0, err = 0.0;
    for (double v : r) mx = fmax(mx, fabs(v));
    for (size_t i = 0; i < r.size(); ++i)
        err = fmax(err, fabs(g[i] - r[i]) / fmax(fmax(fabs(r[i]), 1e-3 * mx), 1e-300));
    return err;
}

int main(int argc, char** argv) {
    if (argc != 6) {
        fprintf(stderr, "usage: %s N C HW dtype seed\n", argv[0]);
        return 2;
    }
    const int64_t N = atoll(argv[1]), C = atoll(argv[2]), HW = atoll(argv[3]);
    const int dtype = atoi(argv[4]);
    Rng rng{static_cast<uint64_t>(atoll(argv[5])) * 2654435761ull + 12345u};
    const size_t E = static_cast<size_t>(N * C * HW), eb = dtype == IABN_F32 ? 4 : 2;
    const float eps = 1e-5f, momentum = 0.1f, slope = 0.01f;

    std::vector<double> mu(C), sd(C), gamma(C), beta(C), x(E), dz(E);
    std::vector<float> g32(C), b32(C), rm(C, 0.f), rv(C, 1.f);
    for (int64_t c = 0; c < C; ++c) {
        mu[c] = -2.0 + 4.0 * rng.uniform();
        sd[c] = 0.5 + 2.5 * rng.uniform();
        g32[c] = static_cast<float>(0.5 + rng.uniform());
        b32[c] = static_cast<float>(0.1 * rng.normal());
        gamma[c] = g32[c];
        beta[c] = b32[c];
    }
    std::vector<uint8_t> xs(E * eb), dzs(E * eb);
    for (size_t i = 0; i < E; ++i) {
        const int64_t c = static_cast<int64_t>((i / HW) % C);
        const uint32_t bx = store(mu[c] + sd[c] * rng.normal(), dtype, &x[i]);
        const uint32_t bd = store(0.1 * rng.normal(), dtype, &dz[i]);
        memcpy(&xs[i * eb], &bx, eb);
        memcpy(&dzs[i * eb], &bd, eb);
    }

    hipStream_t st;
    CHECK_HIP(hipStreamCreate(&st));
    void *dx_z, *ddz, *dws;
    float *dg, *dbt, *drm, *drv, *dsm, *dsv, *ddg, *ddb;
    const size_t ws = iabn_workspace_size(N, C, HW, dtype);
    CHECK_HIP(hipMalloc(&dx_z, E * eb));
    CHECK_HIP(hipMalloc(&ddz, E * eb));
    CHECK_HIP(hipMalloc(&dws, ws > 0 ? ws : 16));
    float** vecs[] = {&dg, &dbt, &drm, &drv, &dsm, &dsv, &ddg, &ddb};
    for (float** p : vecs) CHECK_HIP(hipMalloc(reinterpret_cast<void**>(p), C * sizeof(float)));
    CHECK_HIP(hipMemcpyAsync(dx_z, xs.data(), E * eb, hipMemcpyHostToDevice, st));
    CHECK_HIP(hipMemcpyAsync(ddz, dzs.data(), E * eb, hipMemcpyHostToDevice, st));
    CHECK_HIP(hipMemcpyAsync(dg, g32.data(), C * 4, hipMemcpyHostToDevice, st));
    CHECK_HIP(hipMemcpyAsync(dbt, b32.data(), C * 4, hipMemcpyHostToDevice, st));
    CHECK_HIP(hipMemcpyAsync(drm, rm.data(), C * 4, hipMemcpyHostToDevice, st));
    CHECK_HIP(hipMemcpyAsync(drv, rv.data(), C * 4, hipMemcpyHostToDevice, st));

    // An invalid call first: it must fail on the host and change nothing.
    if (iabn_forward_train(dx_z, dtype, dg, dbt, drm, drv, dsm, dsv, eps, momentum, -1.f, N, C, HW,
                           dws, ws, st) != IABN_ERR_PARAM) {
        fprintf(stderr, "a negative slope was not rejected\n");
        return 1;
    }
    CHECK_IABN(iabn_forward_train(dx_z, dtype, dg, dbt, drm, drv, dsm, dsv, eps, momentum, slope,
                                  N, C, HW, dws, ws, st));
    CHECK_IABN(iabn_backward(dx_z, ddz, dtype, dg, dbt, dsv, ddg, ddb, eps, slope, N, C, HW, dws,
                             ws, st));
    std::vector<uint8_t> zs(E * eb), dxs(E * eb);
    std::vector<float> sm(C), sv(C), rm2(C), rv2(C), dg2(C), db2(C);
    CHECK_HIP(hipMemcpyAsync(zs.data(), dx_z, E * eb, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(dxs.data(), ddz, E * eb, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(sm.data(), dsm, C * 4, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(sv.data(), dsv, C * 4, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(rm2.data(), drm, C * 4, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(rv2.data(), drv, C * 4, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(dg2.data(), ddg, C * 4, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipMemcpyAsync(db2.data(), ddb, C * 4, hipMemcpyDeviceToHost, st));
    CHECK_HIP(hipStreamSynchronize(st));

    // The oracle: forward on x, backward from the GPU-independent stored z
    // (the oracle's z rounded to the storage type), as in the parity tests.
    std::vector<double> z(E), mean(C), var(C), orm(C, 0.0), orv(C, 1.0);
    oracle_forward_train(x.data(), N, C, HW, gamma.data(), beta.data(), eps, momentum, slope,
                         orm.data(), orv.data(), z.data(), mean.data(), var.data());
    std::vector<double> gz(E), gmean(C), gvar(C), grm(C), grv(C);
    for (size_t i = 0; i < E; ++i) gz[i] = load(zs, i, dtype);
    for (int64_t c = 0; c < C; ++c) {
        gmean[c] = sm[c];
        gvar[c] = sv[c];
        grm[c] = rm2[c];
        grv[c] = rv2[c];
    }
    const double tol = dtype == IABN_F32 ? 1e-4 : 2e-2;
    const double ez = max_rel(gz, z), em = max_rel(gmean, mean), ev = max_rel(gvar, var),
                 erm = max_rel(grm, orm), erv = max_rel(grv, orv);
    // Backward: recompute on both sides from the same stored z would need
    // the GPU to run again; instead compare the GPU chain against the
    // oracle's chain on fp32 storage only (16-bit storage rounds z, see the
    // parity tests), and check the invariants for every type.
    std::vector<double> odx(E), odg(C), odb(C);
    oracle_backward_i(z.data(), dz.data(), N, C, HW, gamma.data(), beta.data(), var.data(), eps,
                      slope, odx.data(), odg.data(), odb.data());
    std::vector<double> gdx(E), gdg(C), gdb(C);
    for (size_t i = 0; i < E; ++i) gdx[i] = load(dxs, i, dtype);
    for (int64_t c = 0; c < C; ++c) {
        gdg[c] = dg2[c];
        gdb[c] = db2[c];
    }
    double sum_dx_rel = 0.0;  // per channel |sum dx| against sum |dx| (sum dx = 0 exactly)
    for (int64_t c = 0; c < C; ++c) {
        double s = 0.0, a = 0.0;
        for (int64_t n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const double v = gdx[(n * C + c) * HW + i];
                s += v;
                a += fabs(v);
            }
        sum_dx_rel = fmax(sum_dx_rel, fabs(s) / fmax(a, 1e-300));
    }
    printf("z %.3e mean %.3e var %.3e running_mean %.3e running_var %.3e sum_dx/sum|dx| %.3e",
           ez, em, ev, erm, erv, sum_dx_rel);
    bool ok = ez <= tol && em <= 1e-4 && ev <= 1e-4 && erm <= 1e-4 && erv <= 1e-4 &&
              sum_dx_rel <= (dtype == IABN_F32 ? 1e-5 : 1e-2);
    if (dtype == IABN_F32) {
        const double edx = max_rel(gdx, odx), edg = max_rel(gdg, odg), edb = max_rel(gdb, odb);
        printf(" dx %.3e dgamma %.3e dbeta %.3e", edx, edg, edb);
        ok = ok && edx <= tol && edg <= tol && edb <= tol;
    }
    printf(" -> %s\n", ok ? "ok" : "FAIL");
    for (float** p : vecs) CHECK_HIP(hipFree(*p));
    CHECK_HIP(hipFree(dx_z));
    CHECK_HIP(hipFree(ddz));
    CHECK_HIP(hipFree(dws));
    CHECK_HIP(hipStreamDestroy(st));
    return ok ? 0 : 1;
}
