// Offline plan: exact weight transform, tap-wise power-of-two quantization
// and the alignment / epilogue-width decisions (Sec. III, Sec. III-B), for
// F(4x4,3x3) and F(2x2,3x3).
//
// U = G f G^T with G = Gint / d (Gint integral, Sec. II: d = 24 for F4, 2 for
// F2).  For one tap (a, b), d^2 U = sum_{i,j} Gint[a][i] Gint[b][j] f[i][j];
// every term is an integer of magnitude <= 576 times an fp32 value, hence
// exact in double.  The sum of the nine terms is kept exact as a
// non-overlapping floating-point expansion (Shewchuk, "Adaptive Precision
// Floating-Point Arithmetic and Fast Robust Geometric Predicates", 1997:
// TwoSum and GROW-EXPANSION), which decides every comparison against a
// power-of-two range or a rounding threshold without error.  A double
// approximation of each sum drives the search; the exact expansion is
// consulted only near a decision boundary.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <new>
#include "winof4_internal.h"

using namespace winof4;

namespace {

// Knuth's TwoSum: s + e == a + b exactly, s = fl(a + b).
inline void two_sum(double a, double b, double& s, double& e) {
    s = a + b;
    double bv = s - a;
    double av = s - bv;
    e = (a - av) + (b - bv);
}

// Exact sum of n doubles as a non-overlapping expansion ordered by
// increasing magnitude (zero components dropped).  Returns its length.
int exact_sum(const double* x, int n, double* out) {
    int len = 0;
    double tmp[16];
    for (int k = 0; k < n; ++k) {
        double q = x[k];
        int m = 0;
        for (int i = 0; i < len; ++i) {
            double s, e;
            two_sum(q, out[i], s, e);
            if (e != 0.0) tmp[m++] = e;
            q = s;
        }
        if (q != 0.0) tmp[m++] = q;
        std::memcpy(out, tmp, sizeof(double) * m);
        len = m;
    }
    return len;
}

// Sign of (sum of terms[0..8]) - thr, exactly.
int exact_sign_minus(const double* terms, double thr) {
    double x[10], ex[16];
    std::memcpy(x, terms, sizeof(double) * 9);
    x[9] = -thr;
    int len = exact_sum(x, 10, ex);
    if (len == 0) return 0;
    return ex[len - 1] > 0 ? 1 : -1;   // the largest component carries the sign
}

// The nine exact terms of d^2 * U[a][b] for one 3x3 kernel.
void tap_terms(const Xform& X, const float* f9, int a, int b, double* terms) {
    int k = 0;
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j)
            terms[k++] = (double)(X.gint[a][i] * X.gint[b][j]) * (double)f9[i * 3 + j];
}

// Smallest integer e with |S| <= 2^(bits-1) d^2 2^e over a set of sums
// S = d^2 U, decided exactly.  `approx` holds the double approximation of each
// sum; `terms_of(k, t9)` regenerates the exact terms of sum k.
template <class TermsOf>
int exact_cexp_of_max(const Xform& X, const std::vector<double>& approx, TermsOf terms_of, int bits) {
    const double unit = (double)(1 << (bits - 1)) * X.den2;
    double amax = 0.0;
    for (double v : approx) amax = std::max(amax, std::fabs(v));
    if (amax == 0.0) {
        // approximations are exact zeros only for exact-zero sums (a non-zero
        // expansion never rounds to zero), so the maximum is 0.
        return 0;
    }
    int e;
    std::frexp(amax / unit, &e);     // 2^(e-1) <= amax/unit < 2^e
    e = e - 1;
    if (std::ldexp(unit, e) < amax) e += 1;
    const double rel = 1e-9;
    double t9[9];
    for (int iter = 0; iter < 8; ++iter) {
        bool changed = false;
        // (1) every |S| <= unit * 2^e ?
        double thr = std::ldexp(unit, e);
        for (size_t k = 0; k < approx.size() && !changed; ++k) {
            if (std::fabs(approx[k]) < thr * (1 - rel)) continue;
            terms_of(k, t9);
            if (exact_sign_minus(t9, thr) > 0 || exact_sign_minus(t9, -thr) < 0) {
                e += 1;
                changed = true;
            }
        }
        if (changed) continue;
        // (2) some |S| > unit * 2^(e-1) ?
        double lo = std::ldexp(unit, e - 1);
        bool found = false;
        for (size_t k = 0; k < approx.size() && !found; ++k) {
            double v = std::fabs(approx[k]);
            if (v > lo * (1 + rel)) { found = true; break; }
            if (v < lo * (1 - rel)) continue;
            terms_of(k, t9);
            if (exact_sign_minus(t9, lo) > 0 || exact_sign_minus(t9, -lo) < 0) found = true;
        }
        if (!found) { e -= 1; continue; }
        return e;
    }
    return e;
}

// clamp(R(S / (d^2 2^e)), -2^(bits-1), 2^(bits-1) - 1) for the exact sum S
// of `t9`.
int16_t exact_quantize(const Xform& X, const double* t9, double approx, int e, int bits) {
    const double qmax = (double)((1 << (bits - 1)) - 1), qmin = -(double)(1 << (bits - 1));
    double scale = std::ldexp((double)X.den2, e);
    double u = approx / scale;
    if (!(u < 2.0 * qmax)) return (int16_t)qmax;   // also catches +inf
    if (!(u > 2.0 * qmin)) return (int16_t)qmin;
    double q = std::floor(u + 0.5);
    for (int guard = 0; guard < 4; ++guard) {
        // need (q - 1/2) * scale <= S < (q + 1/2) * scale
        if (exact_sign_minus(t9, (q - 0.5) * scale) < 0) { q -= 1; continue; }
        if (exact_sign_minus(t9, (q + 0.5) * scale) >= 0) { q += 1; continue; }
        break;
    }
    if (q > qmax) q = qmax;
    if (q < qmin) q = qmin;
    return (int16_t)q;
}

}  // namespace

namespace winof4 {

wino_status plan_check_args(const Xform& X, int32_t cin, int32_t cout, const int8_t* in_exp,
                            const int8_t* w_exp, int32_t out_shift, int32_t relu) {
    if (!in_exp) return WINO_EINVAL;
    if (cin < 1 || cout < 1) return WINO_EINVAL;
    if (cin > 65536 || cout > 65536) return WINO_EUNSUPPORTED;
    if (out_shift < 0 || out_shift > 62 || (relu != 0 && relu != 1)) return WINO_EINVAL;
    for (int t = 0; t < X.ntap; ++t) {
        if (in_exp[t] < 0 || in_exp[t] > 15) return WINO_EINVAL;
        if (w_exp && (w_exp[t] < -126 || w_exp[t] > 126)) return WINO_EINVAL;
    }
    return WINO_OK;
}

void plan_set_shape(const Xform& X, wino_f4_plan_s* p, int32_t cin, int32_t cout, int32_t out_shift,
                    int32_t relu) {
    p->m = X.m;
    p->ntap = X.ntap;
    p->cin = cin;
    p->cout = cout;
    p->cin_pad = (int32_t)round_up(cin, kKStep);
    p->cout_pad = (int32_t)round_up(cout, kCoutPad);
    p->out_shift = out_shift;
    p->relu = relu;
}

wino_status plan_finish(const Xform& X, wino_f4_plan_s* p, const int8_t* in_exp, const int32_t* bias,
                        const int32_t* colsum) {
    const int kTaps = X.ntap, n = X.n, cout = p->cout;
    for (int t = 0; t < kTaps; ++t)
        if (p->e_g[t] < -126 || p->e_g[t] > 126) return WINO_ERANGE;
    // exponents and alignment
    int e_o = 1 << 20;
    for (int t = 0; t < kTaps; ++t) {
        p->e_b[t] = in_exp[t];
        e_o = std::min(e_o, (int)in_exp[t] + (int)p->e_g[t]);
    }
    p->e_o = e_o;
    for (int t = 0; t < kTaps; ++t) {
        int s = (int)in_exp[t] + (int)p->e_g[t] - e_o;
        if (s > 62) return WINO_ERANGE;
        p->sh[t] = (int8_t)s;
    }
    // Epilogue bound: max over (co, i, j) of
    //   sum_t |A^T[i][a] A^T[j][b]| 2^sh[t] vmax sum_ci |Uq[t][ci][co]|
    // with vmax = 2^(bits-1) the largest |Vq|
    // plus max|bias| plus the rounding constant.  Every partial sum of the
    // separable output transform is a sub-sum of such a term set, so this
    // bounds all of them.
    int64_t maxbias = 0;
    try {
        p->bias_host.assign(cout, 0);
    } catch (...) {
        return WINO_ENOMEM;
    }
    for (int co = 0; co < cout; ++co) {
        p->bias_host[co] = bias ? bias[co] : 0;
        maxbias = std::max<int64_t>(maxbias, std::llabs((int64_t)p->bias_host[co]));
    }
    unsigned __int128 worst = 0;
    for (int co = 0; co < cout; ++co)
        for (int i = 0; i < X.m; ++i)
            for (int j = 0; j < X.m; ++j) {
                unsigned __int128 tot = 0;
                for (int t = 0; t < kTaps; ++t) {
                    int c = std::abs(X.at[i][t / n] * X.at[j][t % n]);
                    tot += (unsigned __int128)c * (uint32_t)colsum[(size_t)t * cout + co] *
                           (unsigned)(1 << (p->bits - 1)) *
                           ((unsigned __int128)1 << p->sh[t]);
                }
                worst = std::max(worst, tot);
            }
    worst += (unsigned __int128)maxbias;
    if (p->out_shift > 0) worst += (unsigned __int128)1 << (p->out_shift - 1);
    if (worst < ((unsigned __int128)1 << 31) && p->out_shift <= 31) p->epi_bits = 32;
    else if (worst < ((unsigned __int128)1 << 62)) p->epi_bits = 64;
    else return WINO_ERANGE;
    return WINO_OK;
}

wino_status plan_upload_bias(wino_f4_plan_s* p, hipStream_t stream) {
    std::vector<int32_t> bias_pad(p->cout_pad, 0);
    for (int co = 0; co < p->cout; ++co) bias_pad[co] = p->bias_host[co];
    if (hipMalloc(&p->bias_dev, bias_pad.size() * sizeof(int32_t)) != hipSuccess) {
        p->bias_dev = nullptr;
        return WINO_ENOMEM;
    }
    bool ok = hipMemcpyAsync(p->bias_dev, bias_pad.data(), bias_pad.size() * sizeof(int32_t),
                             hipMemcpyHostToDevice, stream) == hipSuccess &&
              hipStreamSynchronize(stream) == hipSuccess;
    return ok ? WINO_OK : WINO_EHIP;
}

}  // namespace winof4

// Host part of the plan: validates the arguments and fills every table of
// `p` (cin, cout, paddings, e_b, e_g, sh, e_o, epi_bits, uq_host, bias_host).
static wino_status compute_tables(const Xform& X, wino_f4_plan_s* p, const float* w_oihw, int32_t cin,
                                  int32_t cout, const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                  int32_t out_shift, int32_t relu, int bits) {
    const int kTaps = X.ntap, n = X.n;
    if (!w_oihw) return WINO_EINVAL;
    wino_status st = plan_check_args(X, cin, cout, in_exp, w_exp, out_shift, relu);
    if (st != WINO_OK) return st;
    for (int64_t i = 0; i < (int64_t)cout * cin * 9; ++i)
        if (!std::isfinite(w_oihw[i])) return WINO_EINVAL;
    plan_set_shape(X, p, cin, cout, out_shift, relu);
    p->bits = bits;

    const int64_t nblk = (int64_t)cout * cin;
    // double approximations of d^2 U for every (block, tap)
    std::vector<double> approx;
    std::vector<int32_t> colsum;
    try {
        approx.resize(nblk * kTaps);
        p->uq_host.assign((size_t)kTaps * cin * cout, 0);
        colsum.assign((size_t)kTaps * cout, 0);
    } catch (...) {
        return WINO_ENOMEM;
    }
    double t9[9], ex[16];
    for (int64_t k = 0; k < nblk; ++k) {
        const float* f9 = w_oihw + k * 9;
        for (int t = 0; t < kTaps; ++t) {
            tap_terms(X, f9, t / n, t % n, t9);
            int len = exact_sum(t9, 9, ex);
            double s = 0.0;
            for (int i = 0; i < len; ++i) s += ex[i];   // small to large
            approx[k * kTaps + t] = s;
        }
    }
    // e_G
    std::vector<double> col(nblk);
    for (int t = 0; t < kTaps; ++t) {
        if (w_exp) {
            p->e_g[t] = w_exp[t];
            continue;
        }
        for (int64_t k = 0; k < nblk; ++k) col[k] = approx[k * kTaps + t];
        int e = exact_cexp_of_max(X, col, [&](size_t kk, double* tt) {
            tap_terms(X, w_oihw + kk * 9, t / n, t % n, tt);
        }, bits);
        if (e < -126 || e > 126) return WINO_ERANGE;
        p->e_g[t] = (int8_t)e;
    }
    // Uq[t][ci][co] and its column sums
    for (int64_t k = 0; k < nblk; ++k) {
        int co = (int)(k / cin), ci = (int)(k % cin);
        for (int t = 0; t < kTaps; ++t) {
            tap_terms(X, w_oihw + k * 9, t / n, t % n, t9);
            int16_t q = exact_quantize(X, t9, approx[k * kTaps + t], p->e_g[t], bits);
            p->uq_host[((size_t)t * cin + ci) * cout + co] = q;
            colsum[(size_t)t * cout + co] += std::abs((int)q);
        }
    }
    return plan_finish(X, p, in_exp, bias, colsum.data());
}

static wino_status plan_tables(const Xform& X, const float* w_oihw, int32_t cin, int32_t cout,
                               const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias, int32_t out_shift,
                               int8_t* e_g, int8_t* sh, int32_t* e_o, int32_t* epilogue_bits, void* uq, int bits) {
    wino_f4_plan_s* p = new (std::nothrow) wino_f4_plan_s();
    if (!p) return WINO_ENOMEM;
    p->uq_dev = nullptr;
    p->bias_dev = nullptr;
    wino_status st = compute_tables(X, p, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, 0, bits);
    if (st == WINO_OK) st = wino_f4_plan_info(p, e_g, sh, e_o, epilogue_bits, nullptr, nullptr, nullptr);
    if (st == WINO_OK && uq) {
        for (size_t i = 0; i < p->uq_host.size(); ++i) {
            if (bits == 10) ((int16_t*)uq)[i] = p->uq_host[i];
            else ((int8_t*)uq)[i] = (int8_t)p->uq_host[i];
        }
    }
    delete p;
    return st;
}

static wino_f4_plan_s* new_plan() {
    wino_f4_plan_s* p = new (std::nothrow) wino_f4_plan_s();
    if (!p) return nullptr;
    p->uq_dev = nullptr;
    p->bias_dev = nullptr;
    return p;
}

static wino_status make_plan(const Xform& X, wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                             const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias, int32_t out_shift,
                             int32_t relu, hipStream_t stream, int bits = 8) {
    if (!out) return WINO_EINVAL;
    *out = nullptr;
    wino_f4_plan_s* p = new_plan();
    if (!p) return WINO_ENOMEM;
    wino_status st = compute_tables(X, p, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, relu, bits);
    if (st != WINO_OK) {
        delete p;
        return st;
    }
    // device upload: Uq k-blocked (GEMM A operand: rows = output channels,
    // one 64-byte k row per row, so one k step of one tap is a single
    // contiguous block), bias [cout_pad]:
    //   bits 8:  int8 [ntap][cin_pad/64][cout_pad][64]
    //   bits 10: fp16 [ntap][cin_pad/32][cout_pad][32] (the 10-bit integers
    //            are exact in fp16; the tap GEMM runs on fp16 matrix cores)
    const int kpr = bits == 10 ? kKStep / 2 : kKStep;        // channels per 64-byte k row
    const int nkb = p->cin_pad / kpr;
    std::vector<int8_t> dev_layout((size_t)X.ntap * p->cout_pad * p->cin_pad * kbytes_per_channel(bits), 0);
    for (int t = 0; t < X.ntap; ++t)
        for (int ci = 0; ci < cin; ++ci)
            for (int co = 0; co < cout; ++co) {
                const size_t idx = (((size_t)t * nkb + ci / kpr) * p->cout_pad + co) * kpr + ci % kpr;
                const int16_t v = p->uq_host[((size_t)t * cin + ci) * cout + co];
                if (bits == 10) {
                    const _Float16 h = (_Float16)v;
                    std::memcpy(dev_layout.data() + 2 * idx, &h, 2);
                } else {
                    dev_layout[idx] = (int8_t)v;
                }
            }
    if (hipGetDevice(&p->device) != hipSuccess) { delete p; return WINO_EHIP; }
    if (hipMalloc(&p->uq_dev, dev_layout.size()) != hipSuccess) { delete p; return WINO_ENOMEM; }
    if (hipMemcpyAsync(p->uq_dev, dev_layout.data(), dev_layout.size(), hipMemcpyHostToDevice, stream) !=
        hipSuccess) {
        wino_f4_plan_destroy(p);
        return WINO_EHIP;
    }
    st = plan_upload_bias(p, stream);    // synchronizes the stream, so dev_layout may go
    if (st != WINO_OK) {
        wino_f4_plan_destroy(p);
        return st;
    }
    *out = p;
    return WINO_OK;
}

// Plans whose weight transform runs on the GPU (fp32 weights on the device,
// or int8 spatial weights with one power-of-two scale).
static wino_status make_plan_device(const Xform& X, wino_f4_plan_t* out, const float* w_f32,
                                    const int8_t* w_i8, int32_t w_scale_exp, int32_t cin, int32_t cout,
                                    const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                    int32_t out_shift, int32_t relu, hipStream_t stream) {
    if (!out) return WINO_EINVAL;
    *out = nullptr;
    if (!w_f32 && !w_i8) return WINO_EINVAL;
    wino_status st = plan_check_args(X, cin, cout, in_exp, w_exp, out_shift, relu);
    if (st != WINO_OK) return st;
    if (w_i8 && (w_scale_exp < -126 || w_scale_exp > 120)) return WINO_EINVAL;
    wino_f4_plan_s* p = new_plan();
    if (!p) return WINO_ENOMEM;
    plan_set_shape(X, p, cin, cout, out_shift, relu);
    if (hipGetDevice(&p->device) != hipSuccess) { delete p; return WINO_EHIP; }
    std::vector<int32_t> colsum;
    st = w_f32 ? device_weight_tables(X, p, w_f32, w_exp, stream, colsum)
               : device_weight_tables_int8(X, p, w_i8, w_scale_exp, w_exp, stream, colsum);
    if (st == WINO_OK) st = plan_finish(X, p, in_exp, bias, colsum.data());
    if (st == WINO_OK) st = plan_upload_bias(p, stream);
    if (st != WINO_OK) {
        wino_f4_plan_destroy(p);
        return st;
    }
    *out = p;
    return WINO_OK;
}

extern "C" wino_status wino_f4_plan_tables(const float* w_oihw, int32_t cin, int32_t cout,
                                           const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                           int32_t out_shift, int8_t* e_g, int8_t* sh, int32_t* e_o,
                                           int32_t* epilogue_bits, int8_t* uq) {
    return plan_tables(kF4, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, e_g, sh, e_o, epilogue_bits, uq, 8);
}

extern "C" wino_status wino_f2_plan_tables(const float* w_oihw, int32_t cin, int32_t cout,
                                           const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                           int32_t out_shift, int8_t* e_g, int8_t* sh, int32_t* e_o,
                                           int32_t* epilogue_bits, int8_t* uq) {
    return plan_tables(kF2, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, e_g, sh, e_o, epilogue_bits, uq, 8);
}

extern "C" wino_status wino_f4_plan_tables_i10(const float* w_oihw, int32_t cin, int32_t cout,
                                               const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                               int32_t out_shift, int8_t* e_g, int8_t* sh, int32_t* e_o,
                                               int32_t* epilogue_bits, int16_t* uq) {
    return plan_tables(kF4, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, e_g, sh, e_o, epilogue_bits, uq, 10);
}

extern "C" wino_status wino_f2_plan_tables_i10(const float* w_oihw, int32_t cin, int32_t cout,
                                               const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                               int32_t out_shift, int8_t* e_g, int8_t* sh, int32_t* e_o,
                                               int32_t* epilogue_bits, int16_t* uq) {
    return plan_tables(kF2, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, e_g, sh, e_o, epilogue_bits, uq, 10);
}

extern "C" wino_status wino_f4_plan_i10(wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                                        const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                        int32_t out_shift, int32_t relu, hipStream_t stream) {
    return make_plan(kF4, out, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, relu, stream, 10);
}

extern "C" wino_status wino_f2_plan_i10(wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                                        const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                        int32_t out_shift, int32_t relu, hipStream_t stream) {
    return make_plan(kF2, out, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, relu, stream, 10);
}

extern "C" wino_status wino_f4_plan(wino_f4_plan_t* out, const float* w_oihw, int32_t cin,
                                    int32_t cout, const int8_t* in_exp, const int8_t* w_exp,
                                    const int32_t* bias, int32_t out_shift, int32_t relu,
                                    hipStream_t stream) {
    return make_plan(kF4, out, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, relu, stream);
}

extern "C" wino_status wino_f2_plan(wino_f4_plan_t* out, const float* w_oihw, int32_t cin,
                                    int32_t cout, const int8_t* in_exp, const int8_t* w_exp,
                                    const int32_t* bias, int32_t out_shift, int32_t relu,
                                    hipStream_t stream) {
    return make_plan(kF2, out, w_oihw, cin, cout, in_exp, w_exp, bias, out_shift, relu, stream);
}

extern "C" wino_status wino_f4_plan_device(wino_f4_plan_t* out, const float* w_oihw_dev, int32_t cin,
                                           int32_t cout, const int8_t* in_exp, const int8_t* w_exp,
                                           const int32_t* bias, int32_t out_shift, int32_t relu,
                                           hipStream_t stream) {
    if (!w_oihw_dev) return WINO_EINVAL;
    return make_plan_device(kF4, out, w_oihw_dev, nullptr, 0, cin, cout, in_exp, w_exp, bias, out_shift, relu,
                            stream);
}

extern "C" wino_status wino_f2_plan_device(wino_f4_plan_t* out, const float* w_oihw_dev, int32_t cin,
                                           int32_t cout, const int8_t* in_exp, const int8_t* w_exp,
                                           const int32_t* bias, int32_t out_shift, int32_t relu,
                                           hipStream_t stream) {
    if (!w_oihw_dev) return WINO_EINVAL;
    return make_plan_device(kF2, out, w_oihw_dev, nullptr, 0, cin, cout, in_exp, w_exp, bias, out_shift, relu,
                            stream);
}

extern "C" wino_status wino_f4_plan_int8(wino_f4_plan_t* out, const int8_t* w_oihw_dev, int32_t w_scale_exp,
                                         int32_t cin, int32_t cout, const int8_t* in_exp, const int8_t* w_exp,
                                         const int32_t* bias, int32_t out_shift, int32_t relu,
                                         hipStream_t stream) {
    if (!w_oihw_dev) return WINO_EINVAL;
    return make_plan_device(kF4, out, nullptr, w_oihw_dev, w_scale_exp, cin, cout, in_exp, w_exp, bias,
                            out_shift, relu, stream);
}

extern "C" wino_status wino_f2_plan_int8(wino_f4_plan_t* out, const int8_t* w_oihw_dev, int32_t w_scale_exp,
                                         int32_t cin, int32_t cout, const int8_t* in_exp, const int8_t* w_exp,
                                         const int32_t* bias, int32_t out_shift, int32_t relu,
                                         hipStream_t stream) {
    if (!w_oihw_dev) return WINO_EINVAL;
    return make_plan_device(kF2, out, nullptr, w_oihw_dev, w_scale_exp, cin, cout, in_exp, w_exp, bias,
                            out_shift, relu, stream);
}

extern "C" void wino_f4_plan_destroy(wino_f4_plan_t p) {
    if (!p) return;
    if (p->uq_dev) hipFree(p->uq_dev);
    if (p->bias_dev) hipFree(p->bias_dev);
    delete p;
}

extern "C" wino_status wino_f4_plan_set_tap_kernel(wino_f4_plan_t p, int32_t kind) {
    if (!p || kind < WINO_TAP_AUTO || kind > WINO_TAP_ROWS_STREAMK) return WINO_EINVAL;
    p->tap_kernel = kind;
    return WINO_OK;
}

extern "C" wino_status wino_f4_plan_info(wino_f4_plan_t p, int8_t* e_g, int8_t* sh, int32_t* e_o,
                                         int32_t* epilogue_bits, int8_t* uq, int32_t* cin,
                                         int32_t* cout) {
    if (!p) return WINO_EINVAL;
    if (uq && p->bits != 8) return WINO_EINVAL;         // 10-bit tables: wino_f4_plan_tables_i10
    if (e_g) std::memcpy(e_g, p->e_g, p->ntap);
    if (sh) std::memcpy(sh, p->sh, p->ntap);
    if (e_o) *e_o = p->e_o;
    if (epilogue_bits) *epilogue_bits = p->epi_bits;
    if (uq) {
        if (!p->uq_host.empty()) {
            for (size_t i = 0; i < p->uq_host.size(); ++i) uq[i] = (int8_t)p->uq_host[i];
        } else {
            // device-built plan: read the k-blocked device copy back
            const int nkb = p->cin_pad / kKStep;
            std::vector<int8_t> dev((size_t)p->ntap * p->cout_pad * p->cin_pad);
            int cur = 0;
            if (hipGetDevice(&cur) != hipSuccess || hipSetDevice(p->device) != hipSuccess) return WINO_EHIP;
            hipError_t e = hipMemcpy(dev.data(), p->uq_dev, dev.size(), hipMemcpyDeviceToHost);
            hipSetDevice(cur);
            if (e != hipSuccess) return WINO_EHIP;
            for (int t = 0; t < p->ntap; ++t)
                for (int ci = 0; ci < p->cin; ++ci)
                    for (int co = 0; co < p->cout; ++co)
                        uq[((size_t)t * p->cin + ci) * p->cout + co] =
                            dev[(((size_t)t * nkb + ci / kKStep) * p->cout_pad + co) * kKStep + ci % kKStep];
        }
    }
    if (cin) *cin = p->cin;
    if (cout) *cout = p->cout;
    return WINO_OK;
}

// Spatial int8 weights of the direct baseline (one power-of-two scale per
// layer).  Each fp32 value v: 73728 * |v| style comparisons are not needed
// here -- v / 2^e is exact in double (power-of-two scaling of a 24-bit
// significand), and R is applied with an exact fractional-part test.
extern "C" wino_status direct_conv_quantize_weights(const float* w_oihw, int32_t cout, int32_t cin,
                                                    int8_t* w_ohwi, int32_t* e_out) {
    if (!w_oihw || !w_ohwi || !e_out || cout < 1 || cin < 1) return WINO_EINVAL;
    int64_t total = (int64_t)cout * cin * 9;
    double amax = 0.0;
    for (int64_t i = 0; i < total; ++i) {
        if (!std::isfinite(w_oihw[i])) return WINO_EINVAL;
        amax = std::max(amax, std::fabs((double)w_oihw[i]));
    }
    int e = 0;
    if (amax > 0.0) {
        // smallest e with amax <= 128 * 2^e; amax is exact, so ldexp tests are exact
        int fe;
        std::frexp(amax / 128.0, &fe);
        e = fe - 1;
        while (std::ldexp(128.0, e) < amax) ++e;
        while (std::ldexp(128.0, e - 1) >= amax) --e;
    }
    for (int co = 0; co < cout; ++co)
        for (int ci = 0; ci < cin; ++ci)
            for (int r = 0; r < 3; ++r)
                for (int c = 0; c < 3; ++c) {
                    double u = std::ldexp((double)w_oihw[((int64_t)(co * cin + ci) * 3 + r) * 3 + c], -e);
                    double fl = std::floor(u);
                    double frac = u - fl;            // exact: u has at most 24 significant bits
                    double q = frac >= 0.5 ? fl + 1.0 : fl;
                    q = std::min(127.0, std::max(-128.0, q));
                    w_ohwi[(((int64_t)co * 3 + r) * 3 + c) * cin + ci] = (int8_t)q;
                }
    *e_out = e;
    return WINO_OK;
}

extern "C" const char* wino_strerror(wino_status s) {
    switch (s) {
        case WINO_OK: return "success";
        case WINO_EINVAL: return "invalid argument";
        case WINO_EUNSUPPORTED: return "size beyond the library's limits";
        case WINO_ERANGE: return "plan tables exceed the integer epilogue range";
        case WINO_ENOMEM: return "out of memory";
        case WINO_EWORKSPACE: return "workspace missing or too small";
        case WINO_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}
