// Sanitizer driver for the host linear algebra of the LoRE fit (lore_fit.cpp's Jacobi
// eigensolver and Cholesky solve), included here so its internal functions are reachable;
// built with -fsanitize=address,undefined together with device_stubs.cpp.  Checks on seeded
// symmetric / SPD matrices of sizes 1..40 (odd and even, for the round-robin bye):
// A = V diag(w) V^T and V V^T = I to 1e-10, and (L L^T) z = b to 1e-10.  Prints "ok".
#include "lore_fit.cpp"

#include <cstdio>

namespace {
uint64_t g_rng = 0x13198A2E03707344ull;
double urand() {
    g_rng ^= g_rng >> 12; g_rng ^= g_rng << 25; g_rng ^= g_rng >> 27;
    return (double)((g_rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0) * 2.0 - 1.0;
}
}  // namespace

int main() {
    int fail = 0;
    for (int n : {1, 2, 3, 4, 7, 8, 15, 16, 31, 40}) {
        std::vector<double> a((size_t)n * n);
        for (int i = 0; i < n; ++i)
            for (int j = 0; j <= i; ++j) a[(size_t)i * n + j] = a[(size_t)j * n + i] = urand();
        if (n > 3) a[1] = a[(size_t)n] = 0.0;  // an entry that starts at zero
        std::vector<double> a0 = a, w, vt;
        jacobi_eigen(n, a, w, vt);
        double err = 0.0, orth = 0.0, scale = 1e-300;
        for (double v : a0) scale = std::fmax(scale, std::fabs(v));
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < n; ++j) {
                double s = 0.0, o = 0.0;
                for (int k = 0; k < n; ++k) {
                    s += vt[(size_t)k * n + i] * w[k] * vt[(size_t)k * n + j];
                    o += vt[(size_t)i * n + k] * vt[(size_t)j * n + k];
                }
                err = std::fmax(err, std::fabs(s - a0[(size_t)i * n + j]));
                orth = std::fmax(orth, std::fabs(o - (i == j ? 1.0 : 0.0)));
            }
        if (err > 1e-10 * scale * n || orth > 1e-10 * n) {
            std::fprintf(stderr, "jacobi n=%d: reconstruction %.3e, orthogonality %.3e\n", n, err, orth);
            fail = 1;
        }
        // SPD: G = M M^T + n I
        std::vector<double> m((size_t)n * n), g((size_t)n * n);
        for (double& v : m) v = urand();
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < n; ++j) {
                double s = i == j ? n : 0.0;
                for (int k = 0; k < n; ++k) s += m[(size_t)i * n + k] * m[(size_t)j * n + k];
                g[(size_t)i * n + j] = s;
            }
        std::vector<double> g0 = g, b(n), z(n);
        for (double& v : b) v = urand();
        z = b;
        if (!cholesky(n, g)) {
            std::fprintf(stderr, "cholesky n=%d: not positive definite\n", n);
            fail = 1;
            continue;
        }
        cholesky_solve(n, g, z.data());
        double res = 0.0;
        for (int i = 0; i < n; ++i) {
            double s = 0.0;
            for (int k = 0; k < n; ++k) s += g0[(size_t)i * n + k] * z[k];
            res = std::fmax(res, std::fabs(s - b[i]));
        }
        if (res > 1e-10 * n) {
            std::fprintf(stderr, "cholesky n=%d: residual %.3e\n", n, res);
            fail = 1;
        }
        // an indefinite matrix is refused
        std::vector<double> neg = g0;
        neg[0] = -1.0;
        if (cholesky(n, neg)) {
            std::fprintf(stderr, "cholesky n=%d accepted an indefinite matrix\n", n);
            fail = 1;
        }
    }
    std::printf(fail ? "FAILED\n" : "ok\n");
    return fail;
}
