// Micro-op handlers of slot programs, shared by the GPU replay kernel and
// the host emulator that checks the scheduler.  Each call executes the
// micro-op of one slot of one lane.
//
// A context type C supplies the lane's register file and memory:
//   double ld(uint32_t f) const;        register named by the low 24 bits of f
//   double ld_raw(uint32_t f) const;    a read whose value may be discarded
//   void st(uint32_t f, double v) const;
//   double obsv(uint32_t i) const;  double param(uint32_t p) const;  double konst(uint32_t i) const;
//   double ckld(uint32_t row) const;  void ckst(uint32_t row, double v) const;
//   void store_loss(double v, bool on) const;  void store_grad(uint32_t p, double v, bool on) const;
//   uint32_t slot() const;
//   static uint32_t uni(uint32_t x);   (a value that is the same in every thread of the wave)
// and W is a payload with members x, y, z, w (this slot's words 0..3) and
// u1(), u2(), u3() (words 1..3 of any slot, whose high bytes hold the
// uniform immediates).
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

// immediates of a payload (uniform)
template <class C, class W>
NDVM_HD uint32_t imm1(const W &p) { return p.u1() >> 24; }
template <class C, class W>
NDVM_HD uint32_t imm2(const W &p) { return p.u2() >> 24; }
template <class C, class W>
NDVM_HD uint32_t imm3(const W &p) { return p.u3() >> 24; }

// base of an adjoint update of register a: +0 on the first contribution
template <class C>
NDVM_HD double base_of(const C &c, uint32_t w0) {
    const double old = c.ld_raw(w0);
    return (w0 & kFirst) ? 0.0 : old;
}

// fma chain of K terms A[x + k sa] * B[y + k sb]; every operand is read
// before the chain starts (K <= 4 unrolled, longer chains in steps of 4)
template <class C>
NDVM_HD double dot_chain(const C &c, uint32_t x, uint32_t y, uint32_t K, uint32_t sa, uint32_t sb) {
    double a[4], b[4];
#pragma unroll
    for (uint32_t k = 0; k < 4; ++k) {
        if (k < K) {
            a[k] = c.ld(x + k * sa);
            b[k] = c.ld(y + k * sb);
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
                a[k] = c.ld(x + (k0 + k) * sa);
                b[k] = c.ld(y + (k0 + k) * sb);
            }
        }
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k)
            if (k0 + k < K) s = fma(a[k], b[k], s);
    }
    return s;
}

// Hot micro-ops (forms below HOT_END): straight-line code, no per-lane
// branches.
template <class C, class W>
NDVM_HD void exec_hot(const C &c, uint32_t form, const W &p) {
    const uint32_t w0 = p.x;
    if (form == MAC) {   // the most frequent form first
        const double x = c.ld(p.y), y = c.ld(p.z), z = c.ld(p.w);
        c.st(w0, x * y + z);
        return;
    }
    switch (form) {
    case ACC: {
        const double x = c.ld(p.y), y = c.ld(p.z), z = c.ld_raw(p.w);
        const double base = (w0 & kFirst) ? 0.0 : z;
        const bool on = (!(w0 & kGated)) | (x != 0.0);
        c.st(w0, on ? base + x * y : base);
        return;
    }
    case MACG: {
        const double x = c.ld(p.y), y = c.ld(p.z), g = c.ld(p.w);
        const double base = base_of(c, w0);
        c.st(w0, g != 0.0 ? base + x * y : base);
        return;
    }
    case DIV:
        c.st(w0, c.ld(p.y) / c.ld(p.z));
        return;
    case ACCD: {
        const double x = c.ld(p.y), y = c.ld(p.z), g = c.ld(p.w);
        const double base = base_of(c, w0);
        c.st(w0, g != 0.0 ? base + x / y : base);
        return;
    }
    case ACCND: {
        const double x = c.ld(p.y), y = c.ld(p.z), g = c.ld(p.w);
        const double base = base_of(c, w0);
        c.st(w0, g != 0.0 ? base + -(x / y) : base);
        return;
    }
    case DOT: {
        const uint32_t i1 = imm1<C>(p);
        c.st(w0, dot_chain(c, p.y, p.z, i1 & 0x7Fu, imm2<C>(p), imm3<C>(p)));
        return;
    }
    case DOTACC: {
        const uint32_t i1 = imm1<C>(p);
        double s = dot_chain(c, p.y, p.z, i1 & 0x7Fu, imm2<C>(p), imm3<C>(p));
        if (i1 & kNegate) s = -s;
        const double g = c.ld(p.w);
        const double base = base_of(c, w0);
        c.st(w0, g != 0.0 ? base + s : base);
        return;
    }
    case CMPLT:
        c.st(w0, c.ld(p.y) < c.ld(p.z) ? 1.0 : 0.0);
        return;
    case SELP: {
        const double q = c.ld(p.y), y = c.ld(p.z), z = c.ld(p.w);
        c.st(w0, q != 0.0 ? y : z);
        return;
    }
    case ACCSEL: {
        const double x = c.ld(p.y), q = c.ld(p.z), g = c.ld(p.w);
        const bool want = imm1<C>(p) != 0;
        const double base = base_of(c, w0);
        c.st(w0, ((g != 0.0) & ((q != 0.0) == want)) ? base + x : base);
        return;
    }
    case DET2: {
        const double a0 = c.ld(p.y), a1 = c.ld(p.y + 1), a2 = c.ld(p.y + 2), a3 = c.ld(p.y + 3);
        const double t1 = a0 * a3;
        const double t2 = a1 * a2;
        c.st(w0, t1 - t2);
        return;
    }
    case NZ: {
        // reads in groups of four; bitwise ors, so no lane skips a read
        const uint32_t K = imm1<C>(p);
        bool nz = false;
        for (uint32_t k0 = 0; k0 < K; k0 += 4) {
            double v[4];
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) v[k] = k0 + k < K ? c.ld(p.y + k0 + k) : 0.0;
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) nz = nz | (v[k] != 0.0);
        }
        c.st(w0, nz ? 1.0 : 0.0);
        return;
    }
    case GATEGT: {
        const double x = c.ld(p.y), y = c.ld(p.z), g = c.ld(p.w);
        c.st(w0, ((g != 0.0) & (x > y)) ? 1.0 : 0.0);
        return;
    }
    case ACCABS: {
        const double x = c.ld(p.y), a = c.ld(p.z), g = c.ld(p.w);
        const double v = a > 0.0 ? x : (a < 0.0 ? -x : 0.0);
        const double base = base_of(c, w0);
        c.st(w0, g != 0.0 ? base + v : base);
        return;
    }
    case SUMK: {
        // reads in groups of four, then the sum in index order
        const uint32_t K = imm1<C>(p), st = imm2<C>(p);
        double s = 0.0;
        for (uint32_t k0 = 0; k0 < K; k0 += 4) {
            double v[4];
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) v[k] = k0 + k < K ? c.ld(p.y + (k0 + k) * st) : 0.0;
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k)
                if (k0 + k < K) s = (k0 + k == 0) ? v[0] : s + v[k];
        }
        c.st(w0, s);
        return;
    }
    case LDOBS:
        c.st(w0, c.obsv(p.y & kFieldMask));
        return;
    case LDPARAM:
        c.st(w0, c.param(p.y & kFieldMask));
        return;
    case LDCONST:
        c.st(w0, c.konst(p.y & kFieldMask));
        return;
    case CKST:
        c.ckst(p.y & kFieldMask, c.ld(w0));
        return;
    case CKLD:
        c.st(w0, c.ckld(p.y & kFieldMask));
        return;
    case ZERO:
        c.st(w0, 0.0);
        return;
    default:
        return;
    }
}

// Cold micro-ops (everything but END, which the caller handles).
template <class C, class W>
NDVM_HD void exec_cold(const C &c, uint32_t form, const W &p) {
    const uint32_t w0 = p.x;
    switch (form) {
    case UN: {
        const double x = c.ld(p.y);
        double r;
        switch (imm1<C>(p)) {
        case U_EXP: r = exp(x); break;
        case U_LOGC: r = log(clampv(x)); break;
        case U_SQRTC: r = sqrt(clampv(x)); break;
        case U_SIN: r = sin(x); break;
        case U_COS: r = cos(x); break;
        case U_ABS: r = fabs(x); break;
        default: r = log(x); break;
        }
        c.st(w0, r);
        return;
    }
    case POW:
        c.st(w0, pow(c.ld(p.y), c.ld(p.z)));
        return;
    case STLOSS:
        c.store_loss(c.ld(w0), c.slot() < imm1<C>(p));
        return;
    case STGRAD:
        c.store_grad(p.y & kFieldMask, c.ld(w0), c.slot() < imm1<C>(p));
        return;
    default:
        return;
    }
}

}  // namespace slotx
}  // namespace ndvm
