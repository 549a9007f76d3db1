// Host-side construction of the block CAT transform and the weight codes.
//
// Off the hot path: runs once per layer after calibration, on the CPU in
// fp64.  Implements Sec. 4 of the paper:
//   eq. 7   M = (Sigma_w # Sigma_x^-1)^(1/2), the alignment-optimal matrix,
//           evaluated per diagonal block of size k;
//   eq. 10  T_b = H_k M_b (block-local normalised Sylvester Hadamard);
// and Sec. 3, eq. 5 for the weights, W' = W T^-1, followed by the
// per-output-channel symmetric quantizer of Sec. 6.
//
// The geometric mean is evaluated in its congruence form
//   Sigma_w # Sigma_x^-1 = Sx^-1/2 (Sx^1/2 Sigma_w Sx^1/2)^1/2 Sx^-1/2
// (the mean is symmetric in its arguments), which needs eigenproblems of
// Sigma_x and of a congruent image of Sigma_w only.  Symmetric
// eigenproblems use the cyclic Jacobi method, which keeps small
// eigenvalues of ill-conditioned calibration blocks accurate.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <exception>
#include <stdexcept>
#include <string>
#include <thread>
#include <vector>

#include "cat_internal.h"

namespace {

using Mat = std::vector<double>;  // square, row-major

constexpr double kEigFloor = 1e-12;

// Cyclic Jacobi: A (n x n, symmetric, destroyed) -> eigenvalues w,
// eigenvectors in the columns of V.
void jacobi_eigh(Mat& A, int n, std::vector<double>& w, Mat& V) {
    V.assign(static_cast<size_t>(n) * n, 0.0);
    for (int i = 0; i < n; ++i) V[static_cast<size_t>(i) * n + i] = 1.0;
    auto at = [&](Mat& M, int r, int c) -> double& {
        return M[static_cast<size_t>(r) * n + c];
    };
    for (int sweep = 0; sweep < 100; ++sweep) {
        // Stop when every off-diagonal entry is negligible relative to the
        // geometric mean of its diagonal pair (relative accuracy criterion).
        bool done = true;
        for (int p = 0; p < n && done; ++p)
            for (int q = p + 1; q < n; ++q) {
                double apq = std::fabs(at(A, p, q));
                double ref = std::sqrt(std::fabs(at(A, p, p)) * std::fabs(at(A, q, q)));
                if (apq > 1e-15 * ref && apq > 1e-300) { done = false; break; }
            }
        if (done) break;
        for (int p = 0; p < n - 1; ++p) {
            for (int q = p + 1; q < n; ++q) {
                const double apq = at(A, p, q);
                const double app = at(A, p, p), aqq = at(A, q, q);
                if (std::fabs(apq) <= 1e-300 ||
                    std::fabs(apq) <= 1e-18 * std::sqrt(std::fabs(app) * std::fabs(aqq))) {
                    at(A, p, q) = 0.0;
                    at(A, q, p) = 0.0;
                    continue;
                }
                // Rotation angle that annihilates A[p][q]: tan solves
                // t^2 + 2 theta t - 1 = 0, take the smaller root.
                const double theta = (aqq - app) / (2.0 * apq);
                const double t = (theta >= 0 ? 1.0 : -1.0) /
                                 (std::fabs(theta) + std::sqrt(theta * theta + 1.0));
                const double c = 1.0 / std::sqrt(t * t + 1.0);
                const double s = t * c;
                // columns p, q of A
                for (int r = 0; r < n; ++r) {
                    const double arp = at(A, r, p), arq = at(A, r, q);
                    at(A, r, p) = c * arp - s * arq;
                    at(A, r, q) = s * arp + c * arq;
                }
                // rows p, q of A
                double* rp = &at(A, p, 0);
                double* rq = &at(A, q, 0);
                for (int r = 0; r < n; ++r) {
                    const double apr = rp[r], aqr = rq[r];
                    rp[r] = c * apr - s * aqr;
                    rq[r] = s * apr + c * aqr;
                }
                at(A, p, q) = 0.0;
                at(A, q, p) = 0.0;
                // accumulate the rotation into V (columns p, q)
                for (int r = 0; r < n; ++r) {
                    const double vrp = at(V, r, p), vrq = at(V, r, q);
                    at(V, r, p) = c * vrp - s * vrq;
                    at(V, r, q) = s * vrp + c * vrq;
                }
            }
        }
    }
    w.resize(n);
    for (int i = 0; i < n; ++i) w[i] = at(A, i, i);
}

// f(S) = V diag(g(lambda)) V^T for symmetric positive definite S, with
// eigenvalues floored at kEigFloor * lambda_max.  Returns two powers at once.
void spd_powers(const Mat& S, int n, double p1, Mat& out1, double p2, Mat* out2) {
    Mat A(S);
    for (int i = 0; i < n; ++i)
        for (int j = i + 1; j < n; ++j) {
            const double v = 0.5 * (A[static_cast<size_t>(i) * n + j] +
                                    A[static_cast<size_t>(j) * n + i]);
            A[static_cast<size_t>(i) * n + j] = v;
            A[static_cast<size_t>(j) * n + i] = v;
        }
    std::vector<double> w;
    Mat V;
    jacobi_eigh(A, n, w, V);
    const double wmax = *std::max_element(w.begin(), w.end());
    if (!(wmax > 0.0)) throw std::runtime_error("block is not positive definite");
    const double floor = kEigFloor * wmax;
    std::vector<double> g1(n), g2(n);
    for (int i = 0; i < n; ++i) {
        const double l = std::max(w[i], floor);
        g1[i] = std::pow(l, p1);
        g2[i] = std::pow(l, p2);
    }
    auto build = [&](const std::vector<double>& g, Mat& out) {
        out.assign(static_cast<size_t>(n) * n, 0.0);
        for (int i = 0; i < n; ++i)
            for (int j = i; j < n; ++j) {
                double acc = 0.0;
                for (int l = 0; l < n; ++l)
                    acc += V[static_cast<size_t>(i) * n + l] * g[l] *
                           V[static_cast<size_t>(j) * n + l];
                out[static_cast<size_t>(i) * n + j] = acc;
                out[static_cast<size_t>(j) * n + i] = acc;
            }
    };
    build(g1, out1);
    if (out2) build(g2, *out2);
}

// C = A B for n x n matrices.
void matmul(const Mat& A, const Mat& B, Mat& C, int n) {
    C.assign(static_cast<size_t>(n) * n, 0.0);
    for (int i = 0; i < n; ++i) {
        double* ci = &C[static_cast<size_t>(i) * n];
        for (int l = 0; l < n; ++l) {
            const double a = A[static_cast<size_t>(i) * n + l];
            const double* bl = &B[static_cast<size_t>(l) * n];
            for (int j = 0; j < n; ++j) ci[j] += a * bl[j];
        }
    }
}

// In place: each column of M (n x n) replaced by H_n column / sqrt(n),
// H_n the Sylvester Hadamard matrix (fast Walsh-Hadamard butterflies).
void hadamard_left(Mat& M, int n) {
    for (int h = 1; h < n; h <<= 1)
        for (int i = 0; i < n; i += 2 * h)
            for (int r = i; r < i + h; ++r) {
                double* a = &M[static_cast<size_t>(r) * n];
                double* b = &M[static_cast<size_t>(r + h) * n];
                for (int j = 0; j < n; ++j) {
                    const double x = a[j], y = b[j];
                    a[j] = x + y;
                    b[j] = x - y;
                }
            }
    const double s = 1.0 / std::sqrt(static_cast<double>(n));
    for (auto& v : M) v *= s;
}

// Inverse by Gauss-Jordan elimination with partial pivoting.
void invert(const Mat& A, Mat& Ainv, int n) {
    Mat a(A);
    Ainv.assign(static_cast<size_t>(n) * n, 0.0);
    for (int i = 0; i < n; ++i) Ainv[static_cast<size_t>(i) * n + i] = 1.0;
    for (int col = 0; col < n; ++col) {
        int piv = col;
        double best = std::fabs(a[static_cast<size_t>(col) * n + col]);
        for (int r = col + 1; r < n; ++r) {
            const double v = std::fabs(a[static_cast<size_t>(r) * n + col]);
            if (v > best) { best = v; piv = r; }
        }
        if (!(best > 0.0)) throw std::runtime_error("transform block is singular");
        if (piv != col)
            for (int j = 0; j < n; ++j) {
                std::swap(a[static_cast<size_t>(piv) * n + j], a[static_cast<size_t>(col) * n + j]);
                std::swap(Ainv[static_cast<size_t>(piv) * n + j], Ainv[static_cast<size_t>(col) * n + j]);
            }
        const double inv = 1.0 / a[static_cast<size_t>(col) * n + col];
        for (int j = 0; j < n; ++j) {
            a[static_cast<size_t>(col) * n + j] *= inv;
            Ainv[static_cast<size_t>(col) * n + j] *= inv;
        }
        for (int r = 0; r < n; ++r) {
            if (r == col) continue;
            const double f = a[static_cast<size_t>(r) * n + col];
            if (f == 0.0) continue;
            for (int j = 0; j < n; ++j) {
                a[static_cast<size_t>(r) * n + j] -= f * a[static_cast<size_t>(col) * n + j];
                Ainv[static_cast<size_t>(r) * n + j] -= f * Ainv[static_cast<size_t>(col) * n + j];
            }
        }
    }
}

// fp64 -> fp32 (round to nearest even) -> bf16 bits (round to nearest even).
uint16_t to_bf16_bits(double v) {
    const float f = static_cast<float>(v);
    uint32_t u;
    std::memcpy(&u, &f, 4);
    const uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return static_cast<uint16_t>(u >> 16);
}

double bf16_bits_to_double(uint16_t b) {
    const uint32_t u = static_cast<uint32_t>(b) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return static_cast<double>(f);
}

struct BuildJob {
    const double* sx;
    const float* W;
    int64_t d_out, d_in;
    int k;
    int flags;
    int t_dtype;
    void* T_out;
    double* T_exact_out;
    double* W_prime_out;
};

void build_block(const BuildJob& job, int64_t b) {
    const int k = job.k;
    const size_t kk = static_cast<size_t>(k) * k;
    const int64_t c0 = b * k;
    Mat T(kk, 0.0);
    if (job.flags & CAT_BUILD_ALIGN) {
        // Sigma_w,b = W[:, b]^T W[:, b] (upper triangle, then mirrored)
        Mat Sw(kk, 0.0);
        std::vector<double> row(k);
        for (int64_t o = 0; o < job.d_out; ++o) {
            const float* wr = job.W + o * job.d_in + c0;
            for (int i = 0; i < k; ++i) row[i] = static_cast<double>(wr[i]);
            for (int i = 0; i < k; ++i) {
                const double ri = row[i];
                if (ri == 0.0) continue;
                double* si = &Sw[static_cast<size_t>(i) * k];
                for (int j = i; j < k; ++j) si[j] += ri * row[j];
            }
        }
        for (int i = 0; i < k; ++i)
            for (int j = i + 1; j < k; ++j)
                Sw[static_cast<size_t>(j) * k + i] = Sw[static_cast<size_t>(i) * k + j];
        const Mat Sx(job.sx + b * kk, job.sx + (b + 1) * kk);
        Mat Sxh, Sxih;
        spd_powers(Sx, k, 0.5, Sxh, -0.5, &Sxih);
        Mat tmp, C, Ch, G;
        matmul(Sxh, Sw, tmp, k);
        matmul(tmp, Sxh, C, k);          // Sx^1/2 Sw Sx^1/2
        spd_powers(C, k, 0.5, Ch, 0.0, nullptr);
        matmul(Sxih, Ch, tmp, k);
        matmul(tmp, Sxih, G, k);         // Sw # Sx^-1
        spd_powers(G, k, 0.5, T, 0.0, nullptr);   // M_b = G^1/2
    } else {
        for (int i = 0; i < k; ++i) T[static_cast<size_t>(i) * k + i] = 1.0;
    }
    if (job.flags & CAT_BUILD_HADAMARD) hadamard_left(T, k);
    if (job.T_exact_out) std::memcpy(job.T_exact_out + b * kk, T.data(), kk * sizeof(double));
    // round to the storage precision; W' uses the rounded values
    Mat Tr(kk);
    if (job.t_dtype == CAT_BF16) {
        uint16_t* out = static_cast<uint16_t*>(job.T_out) + b * kk;
        for (size_t i = 0; i < kk; ++i) {
            out[i] = to_bf16_bits(T[i]);
            Tr[i] = bf16_bits_to_double(out[i]);
        }
    } else {
        float* out = static_cast<float*>(job.T_out) + b * kk;
        for (size_t i = 0; i < kk; ++i) {
            out[i] = static_cast<float>(T[i]);
            Tr[i] = static_cast<double>(out[i]);
        }
    }
    if (job.W_prime_out) {
        Mat Ti;
        invert(Tr, Ti, k);
        std::vector<double> row(k), acc(k);
        for (int64_t o = 0; o < job.d_out; ++o) {
            const float* wr = job.W + o * job.d_in + c0;
            for (int i = 0; i < k; ++i) row[i] = static_cast<double>(wr[i]);
            std::fill(acc.begin(), acc.end(), 0.0);
            for (int l = 0; l < k; ++l) {
                const double a = row[l];
                if (a == 0.0) continue;
                const double* tl = &Ti[static_cast<size_t>(l) * k];
                for (int j = 0; j < k; ++j) acc[j] += a * tl[j];
            }
            std::memcpy(job.W_prime_out + o * job.d_in + c0, acc.data(), k * sizeof(double));
        }
    }
}

}  // namespace

extern "C" int cat_build_transform(const double* sigma_x_blocks, const float* W,
                                   int64_t d_out, int64_t d_in, int64_t k, int flags,
                                   int t_dtype, void* T_out, double* T_exact_out,
                                   double* W_prime_out, int n_threads) {
    using cat::fail;
    if (!T_out) return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: T_out is NULL");
    if (d_in < 1 || d_out < 1) return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: empty layer");
    if (!cat::is_pow2(k) || k > CAT_MAX_BLOCK)
        return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: k must be a power of two <= 512");
    if (d_in % k) return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: d_in % k != 0");
    if (flags & ~CAT_BUILD_CAT) return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: unknown flags");
    if (t_dtype != CAT_F32 && t_dtype != CAT_BF16)
        return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: t_dtype must be CAT_F32 or CAT_BF16");
    if ((flags & CAT_BUILD_ALIGN) && (!sigma_x_blocks || !W))
        return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: alignment needs sigma_x_blocks and W");
    if (W_prime_out && !W) return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: W_prime_out needs W");
    try {
        BuildJob job{sigma_x_blocks, W, d_out, d_in, static_cast<int>(k), flags, t_dtype,
                     T_out, T_exact_out, W_prime_out};
        const int64_t nb = d_in / k;
        int nt = n_threads > 0 ? n_threads : static_cast<int>(std::thread::hardware_concurrency());
        nt = std::max(1, std::min<int>(nt, static_cast<int>(nb)));
        std::vector<std::string> errors(nt);
        std::vector<std::thread> pool;
        for (int t = 0; t < nt; ++t)
            pool.emplace_back([&, t] {
                try {
                    for (int64_t b = t; b < nb; b += nt) build_block(job, b);
                } catch (const std::exception& e) {
                    errors[t] = e.what();
                } catch (...) {
                    errors[t] = "unknown error";
                }
            });
        for (auto& th : pool) th.join();
        for (const auto& e : errors)
            if (!e.empty()) return fail(CAT_ERR_INVALID_ARG, "cat_build_transform: " + e);
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string("cat_build_transform: ") + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, "cat_build_transform: unknown error");
    }
    return CAT_OK;
}

extern "C" int cat_quantize_weights(const double* W_prime, int64_t d_out, int64_t d_in,
                                    int bits, uint8_t* codes_w_out, float* s_w_out) {
    using cat::fail;
    if (!W_prime || !codes_w_out || !s_w_out)
        return fail(CAT_ERR_INVALID_ARG, "cat_quantize_weights: NULL pointer");
    if (d_out < 1 || d_in < 2 || (d_in & 1))
        return fail(CAT_ERR_INVALID_ARG, "cat_quantize_weights: d_out >= 1, d_in even >= 2");
    if (bits != 4 && bits != 6 && bits != 8)
        return fail(CAT_ERR_UNSUPPORTED, "cat_quantize_weights: bits must be 4, 6 or 8");
    const float qmax = static_cast<float>((1 << (bits - 1)) - 1);
    // bits 4: two codes per byte; 6 and 8: one int8 per code
    const int64_t row_out = bits == 4 ? d_in / 2 : d_in;
    std::vector<float> row(static_cast<size_t>(d_in));
    std::vector<int> q(static_cast<size_t>(d_in));
    for (int64_t o = 0; o < d_out; ++o) {
        float amax = 0.0f;
        for (int64_t j = 0; j < d_in; ++j) {
            row[j] = static_cast<float>(W_prime[o * d_in + j]);
            amax = std::max(amax, std::fabs(row[j]));
        }
        uint8_t* out = codes_w_out + o * row_out;
        if (amax == 0.0f) {
            s_w_out[o] = 0.0f;
            std::memset(out, 0, static_cast<size_t>(row_out));
            continue;
        }
        s_w_out[o] = amax / qmax;
        const float inv = qmax / amax;
        for (int64_t j = 0; j < d_in; ++j) {
            const float u = row[j] * inv;
            float r = std::nearbyint(u);
            r = std::min(qmax, std::max(-qmax, r));
            q[j] = static_cast<int>(r);
        }
        if (bits == 4) {
            for (int64_t j = 0; j < d_in; j += 2)
                out[j / 2] = static_cast<uint8_t>((q[j] & 0xF) | ((q[j + 1] & 0xF) << 4));
        } else {
            for (int64_t j = 0; j < d_in; ++j) out[j] = static_cast<uint8_t>(q[j] & 0xFF);
        }
    }
    return CAT_OK;
}

extern "C" int cat_weight_code_sums(const uint8_t* codes_w, int64_t d_out, int64_t d_in,
                                    int32_t* rsum_out) {
    using cat::fail;
    if (!codes_w || !rsum_out) return fail(CAT_ERR_INVALID_ARG, "cat_weight_code_sums: NULL pointer");
    if (d_out < 1 || d_in < 2 || (d_in & 1))
        return fail(CAT_ERR_INVALID_ARG, "cat_weight_code_sums: d_out >= 1, d_in even >= 2");
    for (int64_t o = 0; o < d_out; ++o) {
        const uint8_t* row = codes_w + o * (d_in / 2);
        int64_t sum = 0;
        for (int64_t j = 0; j < d_in / 2; ++j) {
            const int lo = row[j] & 0xF, hi = row[j] >> 4;   // two's complement nibbles
            sum += (lo >= 8 ? lo - 16 : lo) + (hi >= 8 ? hi - 16 : hi);
        }
        rsum_out[o] = static_cast<int32_t>(sum);
    }
    return CAT_OK;
}

extern "C" int cat_sqnr_terms(const float* s_x, int64_t n, int bits_x, const double* sigma_sum_blocks,
                              int64_t d_in, int64_t k, const void* T, int t_dtype,
                              const double* W_prime, int64_t d_out, int bits_w, double sum_y2,
                              double* out) {
    using cat::fail;
    if (!s_x || !sigma_sum_blocks || !T || !W_prime || !out)
        return fail(CAT_ERR_INVALID_ARG, "cat_sqnr_terms: NULL pointer");
    if (n < 1 || d_out < 1 || d_in < 1 || !cat::is_pow2(k) || k > CAT_MAX_BLOCK || d_in % k)
        return fail(CAT_ERR_INVALID_ARG, "cat_sqnr_terms: bad sizes");
    if (t_dtype != CAT_F32 && t_dtype != CAT_BF16)
        return fail(CAT_ERR_INVALID_ARG, "cat_sqnr_terms: bad t_dtype");
    if (bits_x < 2 || bits_x > 8 || bits_w < 2 || bits_w > 8)
        return fail(CAT_ERR_INVALID_ARG, "cat_sqnr_terms: bits must lie in [2, 8]");
    const double qx = static_cast<double>((1 << (bits_x - 1)) - 1);
    const double qw = static_cast<double>((1 << (bits_w - 1)) - 1);
    // E||x'||^2 = (1/n) sum_b tr(T_b S_b T_b^T), S_b the block's second-moment sum
    double tr_sum = 0.0;
    std::vector<double> tb(static_cast<size_t>(k * k));
    for (int64_t b = 0; b < d_in / k; ++b) {
        for (int64_t e = 0; e < k * k; ++e)
            tb[e] = t_dtype == CAT_BF16
                        ? bf16_bits_to_double(static_cast<const uint16_t*>(T)[b * k * k + e])
                        : static_cast<double>(static_cast<const float*>(T)[b * k * k + e]);
        const double* S = sigma_sum_blocks + b * k * k;
        for (int64_t j = 0; j < k; ++j)           // row j of T_b: t_j^T S t_j
            for (int64_t a = 0; a < k; ++a) {
                const double ta = tb[j * k + a];
                if (ta == 0.0) continue;
                double acc = 0.0;
                for (int64_t c = 0; c < k; ++c) acc += S[a * k + c] * tb[j * k + c];
                tr_sum += ta * acc;
            }
    }
    const double ex2 = tr_sum / static_cast<double>(n);
    // E[r(x')^2] with r = 2 amax = 2 qmax s_x (the per-token scale)
    double er2 = 0.0;
    for (int64_t t = 0; t < n; ++t) {
        const double r = 2.0 * qx * static_cast<double>(s_x[t]);
        er2 += r * r;
    }
    er2 /= static_cast<double>(n);
    // C(W') and ||W'||_F^2 over output rows
    double wf2 = 0.0, wr2 = 0.0;
    for (int64_t o = 0; o < d_out; ++o) {
        double amax = 0.0;
        for (int64_t j = 0; j < d_in; ++j) {
            const double v = W_prime[o * d_in + j];
            wf2 += v * v;
            amax = std::max(amax, std::fabs(v));
        }
        wr2 += 4.0 * amax * amax;
    }
    const double cx = ex2 / er2;
    const double cw = wf2 / wr2;
    const double a = (sum_y2 / static_cast<double>(n)) / (wf2 * ex2);   // E||W'x'||^2 = E||Wx||^2
    const double nx = 2.0 * qx, nw = 2.0 * qw;
    const double px = nx * nx * cx, pw = nw * nw * cw;
    const double pred = 12.0 * (1.0 / (1.0 / px + 1.0 / pw)) * a;
    out[0] = cx;
    out[1] = cw;
    out[2] = a;
    out[3] = pred;
    out[4] = 10.0 * std::log10(pred);
    return CAT_OK;
}

namespace {
// Entry (r, c) of the unnormalised Hadamard matrix H_m of the
// full-dimension transform: Sylvester for m a power of two, else
// H_28 (x) Sylvester_(m/28) with H_28 from Paley's second construction
// (q = 13), rows split as r = r1 (m/28) + r2.
int legendre13_h(int a) {
    a = ((a % 13) + 13) % 13;
    return a == 0 ? 0 : (a == 1 || a == 3 || a == 4 || a == 9 || a == 10 || a == 12) ? 1 : -1;
}
int paley28_h(int r, int c) {
    const int i = r / 2, j = c / 2, ri = r % 2, cj = c % 2;
    const int conf = (i == 0 && j == 0) ? 0 : (i == 0 || j == 0) ? 1 : legendre13_h(i - j);
    const int a = (ri == 1 && cj == 1) ? -1 : 1;
    const int b = (ri == 0 && cj == 0) ? 1 : -1;
    return conf * a + (i == j ? b : 0);
}
int hadamard_entry(int64_t m, int64_t r, int64_t c) {
    if ((m & (m - 1)) == 0) return (__builtin_popcountll(r & c) & 1) ? -1 : 1;
    const int64_t m2 = m / 28;
    const int syl = (__builtin_popcountll((r % m2) & (c % m2)) & 1) ? -1 : 1;
    return paley28_h(static_cast<int>(r / m2), static_cast<int>(c / m2)) * syl;
}
}  // namespace

extern "C" int cat_full_hadamard_weights(const double* W_prime, int64_t d_out, int64_t d_in,
                                         int64_t k, double* W_full_out) {
    using cat::fail;
    if (!W_prime || !W_full_out) return fail(CAT_ERR_INVALID_ARG, "cat_full_hadamard_weights: NULL pointer");
    if (d_out < 1 || k < 1 || d_in < k || d_in % k)
        return fail(CAT_ERR_INVALID_ARG, "cat_full_hadamard_weights: bad sizes");
    const int64_t m = d_in / k;
    const bool pow2 = (m & (m - 1)) == 0;
    const bool p28 = m % 28 == 0 && ((m / 28) & (m / 28 - 1)) == 0;
    if (!pow2 && !p28) return fail(CAT_ERR_UNSUPPORTED, "cat_full_hadamard_weights: d_in/k has no Hadamard order here");
    std::vector<double> H(static_cast<size_t>(m * m));
    const double norm = 1.0 / std::sqrt(static_cast<double>(m));
    for (int64_t r = 0; r < m; ++r)
        for (int64_t c = 0; c < m; ++c) H[r * m + c] = hadamard_entry(m, r, c) * norm;
    std::vector<double> v(static_cast<size_t>(m));
    for (int64_t o = 0; o < d_out; ++o) {
        const double* src = W_prime + o * d_in;
        double* dst = W_full_out + o * d_in;
        for (int64_t j = 0; j < k; ++j) {
            for (int64_t b = 0; b < m; ++b) v[b] = src[b * k + j];
            for (int64_t a = 0; a < m; ++a) {
                double acc = 0.0;
                for (int64_t b = 0; b < m; ++b) acc += H[a * m + b] * v[b];
                dst[a * k + j] = acc;
            }
        }
    }
    return CAT_OK;
}
