// Offline 3-bit magnitude quantizer for the 4-bit direction codes.
//
// Paper: Appendix "Coordinate-Magnitude Quantizer for 4-Bit Direction Codes"
// and Prop. "Rotation-induced Beta priors": for a unit direction u uniform on
// S^{m-1}, u_j^2 ~ Beta(1/2, (m-1)/2), so X = |u_j| has density
// proportional to (1 - x^2)^{(m-3)/2} on [0, 1].  Lloyd-Max alternates
// conditional means a[t] = E[X | tau_t <= X < tau_{t+1}] and midpoints
// tau_t = (a[t-1] + a[t]) / 2 until it stops moving.
//
// For m = 8 both integrals have closed forms (x = sin(theta)):
//   F(x) = int_0^x (1-t^2)^{5/2} dt
//        = 5 theta/16 + 15 sin(2 theta)/64 + 3 sin(4 theta)/64 + sin(6 theta)/192
//   G(x) = int_0^x t (1-t^2)^{5/2} dt = (1 - (1-x^2)^{7/2}) / 7
// and a[t] = (G(hi) - G(lo)) / (F(hi) - F(lo)).  The iteration runs in
// binary128 (__float128) to a fixed point far below double precision, and the
// result is rounded to double once.  Compiled by the host C++ compiler; no
// device code.

#include <quadmath.h>

#include <mutex>

namespace pariskv {

namespace {

typedef __float128 q128;

q128 prim_f(q128 x) {
    q128 th = asinq(x);
    return 5 * th / 16 + 15 * sinq(2 * th) / 64 + 3 * sinq(4 * th) / 64 + sinq(6 * th) / 192;
}

q128 prim_g(q128 x) {
    q128 r = 1 - x * x;
    q128 r35 = r * r * r * sqrtq(r);
    return (1 - r35) / 7;
}

struct Table {
    double tau[7];
    double a[8];
};

Table g_table;
std::once_flag g_once;

void derive_m8() {
    q128 tau[9];
    tau[0] = 0;
    tau[8] = 1;
    for (int t = 1; t < 8; ++t) tau[t] = (q128)t / 8;
    q128 a[8];
    q128 F[9], G[9];
    for (int it = 0; it < 20000; ++it) {
        for (int t = 0; t <= 8; ++t) {
            F[t] = prim_f(tau[t]);
            G[t] = prim_g(tau[t]);
        }
        for (int t = 0; t < 8; ++t) a[t] = (G[t + 1] - G[t]) / (F[t + 1] - F[t]);
        q128 delta = 0;
        for (int t = 1; t < 8; ++t) {
            q128 nt = (a[t - 1] + a[t]) / 2;
            q128 d = fabsq(nt - tau[t]);
            if (d > delta) delta = d;
            tau[t] = nt;
        }
        if (delta < (q128)1e-31) break;
    }
    for (int t = 0; t <= 8; ++t) {
        F[t] = prim_f(tau[t]);
        G[t] = prim_g(tau[t]);
    }
    for (int t = 0; t < 8; ++t) g_table.a[t] = (double)((G[t + 1] - G[t]) / (F[t + 1] - F[t]));
    for (int t = 1; t < 8; ++t) g_table.tau[t - 1] = (double)tau[t];
}

}  // namespace

// Returns false for unsupported m.
bool quantizer_table_m8(double* tau, double* a) {
    std::call_once(g_once, derive_m8);
    for (int t = 0; t < 7; ++t) tau[t] = g_table.tau[t];
    for (int t = 0; t < 8; ++t) a[t] = g_table.a[t];
    return true;
}

}  // namespace pariskv
