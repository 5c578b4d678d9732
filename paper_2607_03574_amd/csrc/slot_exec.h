// Micro-op handlers of slot programs, shared by the GPU replay kernel and
// the host emulator that checks the scheduler.  Each call executes the
// micro-op of one slot of one lane.
//
// A context type C supplies the lane's register file and memory; registers
// are named by handles (on the GPU an LDS byte address, on the host an
// index):
//   double ld(R h) const;  double ld_raw(R h) const;  (a read whose value may be discarded)
//   void st(R h, double v) const;  R adv(R h, uint32_t n) const;  (n registers further)
//   double obsv(uint32_t i) const;  double param(uint32_t p) const;  double konst(uint32_t i) const;
//   double ckld(uint32_t row) const;  void ckst(uint32_t row, double v) const;
//   void settle(double v) const;  (a no-op use of v that waits for any load of v to land)
//   void check_written(R h) const;  (the host emulator checks h holds a written value; no-op on the GPU)
//   void skip_arm(bool then_taken, uint32_t imm) const;  (SKIP: this lane's predicate; the context
//       decides, over the lanes that share control, whether the next imm & kSkipCountMask
//       instructions are skipped)
//   void store_loss(double v, bool on) const;  void store_grad(uint32_t p, double v, bool on) const;
//   uint32_t slot() const;
// and W is the payload of this slot's micro-op: register handles a(), x(),
// y(), z(), the raw field ix() (an index), the uniform immediate imm(), this
// slot's first-contribution flag first(), and loaded(), which every hot
// handler calls exactly once, after issuing its operand reads and before
// its arithmetic (the GPU decodes the next instruction there, while the
// reads are in flight; the host emulator checks the count).
//
// Adjoint rules follow Appendix C, table tab:adjoints: contractions are fma
// chains over the summation index in ascending order with a plain product as
// the first term; sqrt/log clamp at 1e-8 with no adjoint at or below it;
// sign(0) = 0; the denominator adjoint of a division is -(g*z)/b; a node whose
// incoming adjoint is zero in every element leaves its inputs' adjoints
// untouched; the first contribution to an adjoint stores 0 + x.
#pragma once
#include <hip/hip_runtime.h>

#include <cmath>

#include "slot.h"

#define NDVM_HD __host__ __device__ __forceinline__

namespace ndvm {
namespace slotx {

using namespace slot;

NDVM_HD double clampv(double x) { return x < 1e-8 ? 1e-8 : x; }

// base of an adjoint update: +0 on the first contribution
template <class C, class R>
NDVM_HD double base_of(const C &c, R t, bool first) {
    const double old = c.ld_raw(t);
    return first ? 0.0 : old;
}

// fma chain of K terms A[x + k sa] * B[y + k sb]; operands read in groups of
// four before their terms are added
template <class C, class R>
NDVM_HD double dot_chain(const C &c, R x, R y, uint32_t K, uint32_t sa, uint32_t sb) {
    double a[4], b[4];
#pragma unroll
    for (uint32_t k = 0; k < 4; ++k) {
        if (k < K) {
            a[k] = c.ld(c.adv(x, k * sa));
            b[k] = c.ld(c.adv(y, k * sb));
        }
    }
    double s = a[0] * b[0];
#pragma unroll
    for (uint32_t k = 1; k < 4; ++k)
        if (k < K) s = fma(a[k], b[k], s);
    for (uint32_t k0 = 4; k0 < K; k0 += 4) {
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k) {
            if (k0 + k < K) {
                a[k] = c.ld(c.adv(x, (k0 + k) * sa));
                b[k] = c.ld(c.adv(y, (k0 + k) * sb));
            }
        }
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k)
            if (k0 + k < K) s = fma(a[k], b[k], s);
    }
    return s;
}

// d = 1 if any of the K registers from x on is nonzero, else 0
template <uint32_t K, class C, class W>
NDVM_HD void any_nonzero(const C &c, const W &p) {
    const auto x = p.x();
    double v[K];
#pragma unroll
    for (uint32_t k = 0; k < K; ++k) v[k] = c.ld(c.adv(x, k));
    p.loaded();
    bool nz = false;
#pragma unroll
    for (uint32_t k = 0; k < K; ++k) nz = nz | (v[k] != 0.0);
    c.st(p.a(), nz ? 1.0 : 0.0);
}

// Block of N <= 4 dot products sharing the X operand: d[j] = chain over
// k < K of X[k] * Y[k][j]; every operand is read before the chains start.
// ACC: the adjoint form (gate register z, base per output, negation).
// Strides in registers: X[k] at x + k*sx, Y[k][j] at y + k*sy + j*sc; when
// kStd they are the row-major ones (sx = 1, sy = N, sc = 1) and known here,
// so register offsets fold into the reads.
template <uint32_t K, uint32_t N, bool ACC, bool kStd, class C, class W>
NDVM_HD void dot_block_kn(const C &c, const W &p, uint32_t sx, uint32_t sy, uint32_t sc, bool neg) {
    if (kStd) {
        sx = 1;
        sy = N;
        sc = 1;
    }
    const auto a = p.a(), x = p.x(), y = p.y();
    double X[K], Y[K][N], base[N];
#pragma unroll
    for (uint32_t k = 0; k < K; ++k) {
        X[k] = c.ld(c.adv(x, k * sx));
#pragma unroll
        for (uint32_t j = 0; j < N; ++j) Y[k][j] = c.ld(c.adv(y, k * sy + j * sc));
    }
    double g = 1.0;
    if (ACC) {
        const bool first = p.first();
        g = c.ld(p.z());
#pragma unroll
        for (uint32_t j = 0; j < N; ++j) base[j] = base_of(c, c.adv(a, j), first);
    }
    // the next instruction's decode after the products (with all operands
    // live it would cost registers the wave does not have)
    double out[N];
#pragma unroll
    for (uint32_t j = 0; j < N; ++j) {
        double s = X[0] * Y[0][j];
#pragma unroll
        for (uint32_t k = 1; k < K; ++k) s = fma(X[k], Y[k][j], s);
        if (ACC) {
            if (neg) s = -s;
            s = g != 0.0 ? base[j] + s : base[j];
        }
        out[j] = s;
    }
    p.loaded();
#pragma unroll
    for (uint32_t j = 0; j < N; ++j) c.st(c.adv(a, j), out[j]);
}

// any K, N <= 7: the same arithmetic with uniform loop bounds
template <bool ACC, class C, class W>
NDVM_HD void dot_block_generic(const C &c, const W &p, uint32_t K, uint32_t N, uint32_t sx, uint32_t sy,
                               uint32_t sc, bool neg) {
    p.loaded();
    const auto a = p.a(), x = p.x(), y = p.y();
    const double g = ACC ? c.ld(p.z()) : 1.0;
    const bool first = p.first();
    for (uint32_t j = 0; j < N; ++j) {
        double s = c.ld(x) * c.ld(c.adv(y, j * sc));
        for (uint32_t k = 1; k < K; ++k) s = fma(c.ld(c.adv(x, k * sx)), c.ld(c.adv(y, k * sy + j * sc)), s);
        if (ACC) {
            if (neg) s = -s;
            const double b = base_of(c, c.adv(a, j), first);
            s = g != 0.0 ? b + s : b;
        }
        c.st(c.adv(a, j), s);
    }
}

// Shapes with sides 1, 2 and 4 unrolled; others through the generic loops.
// The forward form takes the row-major strides unrolled too (the layout the
// scheduler gives forward products), the adjoint form its strides at run time.
template <bool ACC, class C, class W>
NDVM_HD void dot_block(const C &c, const W &p) {
    const uint32_t im = p.imm();
    const uint32_t K = im & 7u, N = (im >> 3) & 7u, sx = (im >> 6) & 7u, sy = (im >> 9) & 7u,
                   sc = (im >> 12) & 7u;
    const bool neg = (im >> 15) & 1u;
    const bool std_layout = !ACC && (K == 1 || sy == N) && (N == 1 || sc == 1) && (K == 1 || sx == 1);
    if (std_layout) {
        switch (K * 8 + N) {
#define NDVM_KN(k, n) \
    case k * 8 + n: dot_block_kn<k, n, ACC, true>(c, p, sx, sy, sc, neg); return;
        NDVM_KN(1, 1) NDVM_KN(1, 2) NDVM_KN(1, 4)
        NDVM_KN(2, 1) NDVM_KN(2, 2) NDVM_KN(2, 4)
        NDVM_KN(4, 1) NDVM_KN(4, 2) NDVM_KN(4, 4)
#undef NDVM_KN
        default: break;
        }
    } else if (ACC) {
        switch (K * 8 + N) {
#define NDVM_KN(k, n) \
    case k * 8 + n: dot_block_kn<k, n, ACC, false>(c, p, sx, sy, sc, neg); return;
        NDVM_KN(1, 1) NDVM_KN(1, 2) NDVM_KN(1, 4)
        NDVM_KN(2, 1) NDVM_KN(2, 2) NDVM_KN(2, 4)
        NDVM_KN(4, 1) NDVM_KN(4, 2) NDVM_KN(4, 4)
#undef NDVM_KN
        default: break;
        }
    }
    dot_block_generic<ACC>(c, p, K, N, sx, sy, sc, neg);
}

// The most frequent forms, also callable on their own (the kernel tests for
// them ahead of the general dispatch).
template <class C, class W>
NDVM_HD void exec_mac(const C &c, const W &p) {
    const double x = c.ld(p.x()), y = c.ld(p.y()), z = c.ld(p.z());
    p.loaded();
    c.st(p.a(), x * y + z);
}
template <class C, class W>
NDVM_HD void exec_acc(const C &c, const W &p) {
    const double x = c.ld(p.x()), y = c.ld(p.y()), base = c.ld(p.z());
    p.loaded();
    c.st(p.a(), x != 0.0 ? base + x * y : base);
}
template <class C, class W>
NDVM_HD void exec_msub(const C &c, const W &p) {
    const double x = c.ld(p.x()), y = c.ld(p.y()), z = c.ld(p.z());
    p.loaded();
    c.st(p.a(), x * y - z);
}

// Hot micro-ops (forms below HOT_END): straight-line code, no per-lane
// branches.
template <class C, class W>
NDVM_HD void exec_hot(const C &c, uint32_t form, const W &p) {
    switch (form) {
    case MAC:
        exec_mac(c, p);
        return;
    case ACC:
        exec_acc(c, p);
        return;
    case MACG: {
        const auto a = p.a();
        const double x = c.ld(p.x()), y = c.ld(p.y()), g = c.ld(p.z());
        const double base = base_of(c, a, p.first());
        p.loaded();
        c.st(a, g != 0.0 ? base + x * y : base);
        return;
    }
    case DIV: {
        const double x = c.ld(p.x()), y = c.ld(p.y());
        p.loaded();
        c.st(p.a(), x / y);
        return;
    }
    case MSUB: exec_msub(c, p); return;
    case RSUB: {
        const double x = c.ld(p.x()), y = c.ld(p.y()), z = c.ld(p.z());
        p.loaded();
        c.st(p.a(), z - x * y);
        return;
    }
    case ACCD: {
        const auto a = p.a();
        const double x = c.ld(p.x()), y = c.ld(p.y()), g = c.ld(p.z());
        const double base = base_of(c, a, p.first());
        p.loaded();
        c.st(a, g != 0.0 ? base + x / y : base);
        return;
    }
    case ACCND: {
        const auto a = p.a();
        const double x = c.ld(p.x()), y = c.ld(p.y()), g = c.ld(p.z());
        const double base = base_of(c, a, p.first());
        p.loaded();
        c.st(a, g != 0.0 ? base + -(x / y) : base);
        return;
    }
    case DOT: {
        p.loaded();
        const uint32_t im = p.imm();
        c.st(p.a(), dot_chain(c, p.x(), p.y(), im & 31u, (im >> 6) & 63u, (im >> 12) & 63u));
        return;
    }
    case DOTACC: {
        p.loaded();
        const uint32_t im = p.imm();
        const auto a = p.a();
        double s = dot_chain(c, p.x(), p.y(), im & 31u, (im >> 6) & 63u, (im >> 12) & 63u);
        if ((im >> 5) & 1u) s = -s;
        const double g = c.ld(p.z());
        const double base = base_of(c, a, p.first());
        c.st(a, g != 0.0 ? base + s : base);
        return;
    }
    case CMPLT: {
        const double x = c.ld(p.x()), y = c.ld(p.y());
        p.loaded();
        c.st(p.a(), x < y ? 1.0 : 0.0);
        return;
    }
    case SELP: {   // the untaken arm's register may hold anything (its arm may have been skipped)
        const double q = c.ld(p.x()), y = c.ld_raw(p.y()), z = c.ld_raw(p.z());
        p.loaded();
        c.check_written(q != 0.0 ? p.y() : p.z());
        c.st(p.a(), q != 0.0 ? y : z);
        return;
    }
    case SKIP: {   // wave-level branch skipping: every lane takes the other arm
        const double q = c.ld(p.x());
        p.loaded();
        c.skip_arm(q != 0.0, p.imm());
        return;
    }
    case ACCSEL: {
        const auto a = p.a();
        const double x = c.ld(p.x()), q = c.ld(p.y()), g = c.ld(p.z());
        const bool want = (p.imm() & 1u) != 0;
        const double base = base_of(c, a, p.first());
        p.loaded();
        c.st(a, ((g != 0.0) & ((q != 0.0) == want)) ? base + x : base);
        return;
    }
    case DET2: {
        const auto x = p.x();
        const double a0 = c.ld(x), a1 = c.ld(c.adv(x, 1)), a2 = c.ld(c.adv(x, 2)), a3 = c.ld(c.adv(x, 3));
        p.loaded();
        const double t1 = a0 * a3;
        const double t2 = a1 * a2;
        c.st(p.a(), t1 - t2);
        return;
    }
    case NZ: {
        const uint32_t K = p.imm();
        switch (K) {   // the sizes of small matrices unrolled: every read issued at once
        case 1: any_nonzero<1>(c, p); return;
        case 2: any_nonzero<2>(c, p); return;
        case 4: any_nonzero<4>(c, p); return;
        case 8: any_nonzero<8>(c, p); return;
        case 16: any_nonzero<16>(c, p); return;
        default: break;
        }
        // other sizes: reads in groups of four; bitwise ors, so no lane skips a read
        p.loaded();
        const auto x = p.x();
        bool nz = false;
        for (uint32_t k0 = 0; k0 < K; k0 += 4) {
            double v[4];
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) v[k] = k0 + k < K ? c.ld(c.adv(x, k0 + k)) : 0.0;
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) nz = nz | (v[k] != 0.0);
        }
        c.st(p.a(), nz ? 1.0 : 0.0);
        return;
    }
    case GATEGT: {
        const double x = c.ld(p.x()), y = c.ld(p.y()), g = c.ld(p.z());
        p.loaded();
        c.st(p.a(), ((g != 0.0) & (x > y)) ? 1.0 : 0.0);
        return;
    }
    case ACCABS: {
        const auto a = p.a();
        const double x = c.ld(p.x()), v = c.ld(p.y()), g = c.ld(p.z());
        const double d = v > 0.0 ? x : (v < 0.0 ? -x : 0.0);
        const double base = base_of(c, a, p.first());
        p.loaded();
        c.st(a, g != 0.0 ? base + d : base);
        return;
    }
    case SUMK: {
        // reads in groups of four, then the sum in index order
        p.loaded();
        const uint32_t im = p.imm(), K = im & 63u, st = (im >> 6) & 63u;
        const auto x = p.x();
        double s = 0.0;
        for (uint32_t k0 = 0; k0 < K; k0 += 4) {
            double v[4];
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) v[k] = k0 + k < K ? c.ld(c.adv(x, (k0 + k) * st)) : 0.0;
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k)
                if (k0 + k < K) s = (k0 + k == 0) ? v[0] : s + v[k];
        }
        c.st(p.a(), s);
        return;
    }
    case ZERO:
        p.loaded();
        c.st(p.a(), 0.0);
        return;
    case DOTB:
        dot_block<false>(c, p);
        return;
    case DOTBACC:
        dot_block<true>(c, p);
        return;
    case EXPF: {
        const double x = c.ld(p.x());
        p.loaded();
        c.st(p.a(), exp(x));
        return;
    }
    case LOGCF: {
        const double x = c.ld(p.x());
        p.loaded();
        c.st(p.a(), log(clampv(x)));
        return;
    }
    case LOGF: {
        const double x = c.ld(p.x());
        p.loaded();
        c.st(p.a(), log(x));
        return;
    }
    case SQRTCF: {
        const double x = c.ld(p.x());
        p.loaded();
        c.st(p.a(), sqrt(clampv(x)));
        return;
    }
    case ABSF: {
        const double x = c.ld(p.x());
        p.loaded();
        c.st(p.a(), fabs(x));
        return;
    }

    case LDOBS: {
        const double v = c.obsv(p.ix());
        p.loaded();
        c.st(p.a(), v);
        return;
    }
    case LDPARAM: {
        const double v = c.param(p.ix());
        p.loaded();
        c.st(p.a(), v);
        return;
    }
    case LDCONST: {
        const double v = c.konst(p.ix());
        p.loaded();
        c.st(p.a(), v);
        return;
    }
    case CKST: {   // all loads issued before the first store
        const uint32_t m = p.imm(), f = p.ix(), row = f & kCkRowMask, n1 = f >> kCkRowBits;
        const auto a = p.a();
        double v[kMaxCk];
#pragma unroll
        for (uint32_t k = 0; k < kMaxCk; ++k)
            if (k < m) v[k] = c.ld(c.adv(a, k < n1 ? k : n1));
        p.loaded();
#pragma unroll
        for (uint32_t k = 0; k < kMaxCk; ++k)
            if (k < m) c.ckst(row + (k < n1 ? k : n1), v[k]);
#pragma unroll
        for (uint32_t k = 0; k < kMaxCk; ++k) c.settle(v[k]);
        return;
    }
    case CKLD: {   // all loads issued before the first write
        const uint32_t m = p.imm(), f = p.ix(), row = f & kCkRowMask, n1 = f >> kCkRowBits;
        const auto a = p.a();
        double v[kMaxCk];
#pragma unroll
        for (uint32_t k = 0; k < kMaxCk; ++k)
            if (k < m) v[k] = c.ckld(row + (k < n1 ? k : n1));
        p.loaded();
#pragma unroll
        for (uint32_t k = 0; k < kMaxCk; ++k)
            if (k < m) c.st(c.adv(a, k < n1 ? k : n1), v[k]);
        // every path leaves with all loads landed, so the next handler does
        // not wait for the program prefetch before its own register reads
#pragma unroll
        for (uint32_t k = 0; k < kMaxCk; ++k) c.settle(v[k]);
        return;
    }
    default:
        p.loaded();
        return;
    }
}

// Cold micro-ops (everything but END, which the caller handles): sine,
// cosine, pow, loss and gradient stores.
template <class C, class W>
NDVM_HD void exec_cold(const C &c, uint32_t form, const W &p) {
    switch (form) {
    case UN: {
        const double x = c.ld(p.x());
        c.st(p.a(), p.imm() == U_SIN ? sin(x) : cos(x));
        return;
    }
    case POWF:
        c.st(p.a(), pow(c.ld(p.x()), c.ld(p.y())));
        return;
    case STLOSS:
        c.store_loss(c.ld(p.a()), c.slot() < p.imm());
        return;
    case STGRAD:
        c.store_grad(p.ix(), c.ld(p.a()), c.slot() < p.imm());
        return;
    default:
        return;
    }
}

}  // namespace slotx
}  // namespace ndvm
