// Instruction handlers of the device program, shared by the GPU replay
// kernel and the host-side emulator used to check the scheduler.
//
// A context type C supplies the lane's register file and memory:
//   double ld(uint32_t r) const;  void st(uint32_t r, double v) const;
//   double ld_raw(uint32_t r) const;   (a read whose value may be discarded)
//   double konst(uint32_t i) const;  double obsv(uint32_t i) const;  (uniform loads)
//   static uint32_t uni(uint32_t x);          (wave-uniform value)
//   Fetch prefetch(const uint32_t *pc);  void decode(const Fetch&, uint32_t (&w)[8]);
//   double param(uint32_t p) const;  void store_loss(double) const;
//   void store_grad(uint32_t p, double) const;
//   void ckpt_st(uint32_t row, double) const;  double ckpt_ld(uint32_t row) const;
//
// Adjoint rules follow Appendix C, table tab:adjoints, with these readings:
// contractions are fma chains over the summation index in ascending order
// (first term a plain product); sqrt/log clamp at 1e-8 with no adjoint at or
// below it; sign(0) = 0; the denominator adjoint of a division is g*z/b; a
// node whose incoming adjoint is zero in every element leaves its inputs'
// adjoints untouched (the gating that keeps an untaken select arm from
// producing 0*inf); the first contribution to an adjoint stores 0 + x.
#pragma once
#include <hip/hip_runtime.h>

#include <cmath>

#include "isa.h"

#define NDVM_HD __host__ __device__ __forceinline__

namespace ndvm {
namespace replay {

using namespace isa;

// operand words are register indices
template <class C>
NDVM_HD double opnd(const C &c, uint32_t w) {
    return c.ld(w);
}
// element i of a register operand
template <class C>
NDVM_HD double elem(const C &c, uint32_t w, uint32_t i) {
    return c.ld(w + i);
}
// adjoint update of element i of target word tw with contribution x when
// `on` holds for this lane; the first contribution stores (0 + x)
template <class C>
NDVM_HD void acc(const C &c, uint32_t tw, uint32_t i, double x, bool on) {
    if (tw == kNone) return;
    uint32_t r = (tw & ~kInit) + i;
    if (tw & kInit) {
        c.st(r, on ? 0.0 + x : 0.0);
    } else {
        double v = c.ld(r);
        c.st(r, on ? v + x : v);
    }
}

NDVM_HD double clampv(double x) { return x < 1e-8 ? 1e-8 : x; }

// load an m x n row-major matrix stored at consecutive registers into M[i*4+j]
template <class C>
NDVM_HD void load_mat(const C &c, uint32_t base, uint32_t m, uint32_t n, double (&M)[16]) {
#pragma unroll
    for (uint32_t i = 0; i < 4; ++i)
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) M[i * 4 + j] = (i < m && j < n) ? c.ld(base + i * n + j) : 0.0;
}

NDVM_HD double det2(const double (&A)[16], uint32_t sz) {
    if (sz == 1) return A[0];
    double t1 = A[0] * A[5];
    double t2 = A[1] * A[4];
    return t1 - t2;
}
// inverse (adjugate times r = 1/det), packed into Ai[i*4+j]
NDVM_HD void inv2(const double (&A)[16], uint32_t sz, double (&Ai)[16]) {
#pragma unroll
    for (int i = 0; i < 16; ++i) Ai[i] = 0.0;
    if (sz == 1) {
        Ai[0] = 1.0 / A[0];
        return;
    }
    double r = 1.0 / det2(A, 2);
    Ai[0] = A[5] * r;
    Ai[1] = (-A[1]) * r;
    Ai[4] = (-A[4]) * r;
    Ai[5] = A[0] * r;
}

template <class C>
NDVM_HD bool any_nz(const C &c, uint32_t g, uint32_t n) {
    bool nz = false;
    for (uint32_t i = 0; i < n; ++i) nz = nz || (c.ld(g + i) != 0.0);
    return nz;
}

NDVM_HD double unary_fwd(uint32_t op, double x) {
    switch (op) {
    case F_NEG: return -x;
    case F_EXP: return exp(x);
    case F_LOG: return log(clampv(x));
    case F_SQRT: return sqrt(clampv(x));
    case F_SIN: return sin(x);
    case F_COS: return cos(x);
    default: return fabs(x);
    }
}

template <class C>
NDVM_HD void exec_fwd(const C &c, const uint32_t *aux, const uint32_t *w) {
    const uint32_t op = w[0] & 0xFF, mode = (w[0] >> 8) & 0xFF, n = (w[0] >> 16) & 0xFF;
    const uint32_t dst = w[1];
    switch (op) {
    case F_ADD: case F_SUB: case F_MUL: case F_DIV: {
        for (uint32_t i = 0; i < n; ++i) {
            double x = mode == MODE_A_SCALAR ? opnd(c, w[2]) : elem(c, w[2], i);
            double y = mode == MODE_B_SCALAR ? opnd(c, w[3]) : elem(c, w[3], i);
            double z = op == F_ADD ? x + y : op == F_SUB ? x - y : op == F_MUL ? x * y : x / y;
            c.st(dst + i, z);
        }
        break;
    }
    case F_NEG: case F_EXP: case F_LOG: case F_SQRT: case F_SIN: case F_COS: case F_ABS:
        for (uint32_t i = 0; i < n; ++i) c.st(dst + i, unary_fwd(op, elem(c, w[2], i)));
        break;
    case F_POW:
        c.st(dst, pow(opnd(c, w[2]), opnd(c, w[3])));
        break;
    case F_DOT: {
        double s = elem(c, w[2], 0) * elem(c, w[3], 0);
        for (uint32_t i = 1; i < n; ++i) s = fma(elem(c, w[2], i), elem(c, w[3], i), s);
        c.st(dst, s);
        break;
    }
    case F_MATMUL: {
        const uint32_t m = w[7] & 0xFF, k = (w[7] >> 8) & 0xFF, q = (w[7] >> 16) & 0xFF;
        double A[16], B[16];
        load_mat(c, w[2], m, k, A);
        load_mat(c, w[3], k, q, B);
#pragma unroll
        for (uint32_t i = 0; i < 4; ++i)
#pragma unroll
            for (uint32_t j = 0; j < 4; ++j) {
                if (i < m && j < q) {
                    double s = A[i * 4] * B[j];
#pragma unroll
                    for (uint32_t p = 1; p < 4; ++p)
                        if (p < k) s = fma(A[i * 4 + p], B[p * 4 + j], s);
                    c.st(dst + i * q + j, s);
                }
            }
        break;
    }
    case F_TRANSPOSE: {
        const uint32_t m = w[7] & 0xFF, q = (w[7] >> 8) & 0xFF;   // input m x q
        for (uint32_t i = 0; i < m; ++i)
            for (uint32_t j = 0; j < q; ++j) c.st(dst + j * m + i, c.ld(w[2] + i * q + j));
        break;
    }
    case F_TRACE: {
        const uint32_t sz = w[7];
        double s = c.ld(w[2]);
        for (uint32_t i = 1; i < sz; ++i) s = s + c.ld(w[2] + i * sz + i);
        c.st(dst, s);
        break;
    }
    case F_INV: case F_DET: case F_LOGDET: {
        const uint32_t sz = w[7];
        double A[16], Ai[16];
        load_mat(c, w[2], sz, sz, A);
        if (op == F_INV) {
            inv2(A, sz, Ai);
#pragma unroll
            for (uint32_t i = 0; i < 2; ++i)
#pragma unroll
                for (uint32_t j = 0; j < 2; ++j)
                    if (i < sz && j < sz) c.st(dst + i * sz + j, Ai[i * 4 + j]);
        } else {
            double d = det2(A, sz);
            c.st(dst, op == F_DET ? d : log(clampv(d)));
        }
        break;
    }
    case F_OUTER: {
        const uint32_t m = w[7] & 0xFF, q = (w[7] >> 8) & 0xFF;
        for (uint32_t i = 0; i < m; ++i) {
            double a = elem(c, w[2], i);
            for (uint32_t j = 0; j < q; ++j) c.st(dst + i * q + j, a * elem(c, w[3], j));
        }
        break;
    }
    case F_PACK:
        for (uint32_t i = 0; i < n; ++i) c.st(dst + i, opnd(c, C::aux_word(aux, w[7] + i)));
        break;
    case F_INDEX:
        c.st(dst, c.ld(w[2] + w[7]));
        break;
    case F_SELECT: {
        const bool p = opnd(c, w[2]) < opnd(c, w[3]);
        for (uint32_t i = 0; i < n; ++i) {
            double x = elem(c, w[4], i), y = elem(c, w[5], i);
            c.st(dst + i, p ? x : y);
        }
        break;
    }
    default:
        break;
    }
}

template <class C>
NDVM_HD void exec_rev(const C &c, const uint32_t *aux, const uint32_t *w) {
    const uint32_t op = w[0] & 0xFF, mode = (w[0] >> 8) & 0xFF, n = (w[0] >> 16) & 0xFF;
    const uint32_t g = w[1], ta = w[5], tb = w[6];
    switch (op) {
    case R_ADD: case R_SUB: {
        const bool nz = any_nz(c, g, n);
        for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, c.ld(g + i), nz);
        for (uint32_t i = 0; i < n; ++i) {
            double gi = c.ld(g + i);
            acc(c, tb, i, op == R_ADD ? gi : -gi, nz);
        }
        break;
    }
    case R_MUL: {
        const bool nz = any_nz(c, g, n);
        if (mode == MODE_SAME) {
            for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, c.ld(g + i) * elem(c, w[3], i), nz);
            for (uint32_t i = 0; i < n; ++i) acc(c, tb, i, c.ld(g + i) * elem(c, w[2], i), nz);
        } else if (mode == MODE_A_SCALAR) {   // z = s * M
            double s = c.ld(g) * elem(c, w[3], 0);
            for (uint32_t i = 1; i < n; ++i) s = fma(c.ld(g + i), elem(c, w[3], i), s);
            acc(c, ta, 0, s, nz);
            const double a = opnd(c, w[2]);
            for (uint32_t i = 0; i < n; ++i) acc(c, tb, i, c.ld(g + i) * a, nz);
        } else {                             // z = M * s
            const double b = opnd(c, w[3]);
            for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, c.ld(g + i) * b, nz);
            double s = c.ld(g) * elem(c, w[2], 0);
            for (uint32_t i = 1; i < n; ++i) s = fma(c.ld(g + i), elem(c, w[2], i), s);
            acc(c, tb, 0, s, nz);
        }
        break;
    }
    case R_DIV: {
        const bool nz = any_nz(c, g, n);
        if (mode == MODE_SAME) {
            for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, c.ld(g + i) / elem(c, w[3], i), nz);
            for (uint32_t i = 0; i < n; ++i)
                acc(c, tb, i, -((c.ld(g + i) * elem(c, w[4], i)) / elem(c, w[3], i)), nz);
        } else {                             // z = M / s
            const double b = opnd(c, w[3]);
            for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, c.ld(g + i) / b, nz);
            double s = c.ld(g) * c.ld(w[4]);
            for (uint32_t i = 1; i < n; ++i) s = fma(c.ld(g + i), c.ld(w[4] + i), s);
            acc(c, tb, 0, -(s / b), nz);
        }
        break;
    }
    case R_NEG: case R_EXP: case R_LOG: case R_SQRT: case R_SIN: case R_COS: case R_ABS: {
        const bool nz = any_nz(c, g, n);
        for (uint32_t i = 0; i < n; ++i) {
            const double gi = c.ld(g + i);
            double x = 0.0;
            bool on = nz;
            switch (op) {
            case R_NEG: x = -gi; break;
            case R_EXP: x = gi * c.ld(w[4] + i); break;
            case R_LOG: {
                const double a = elem(c, w[2], i);
                on = on && a > 1e-8;
                x = gi / a;
                break;
            }
            case R_SQRT: {
                const double a = elem(c, w[2], i);
                on = on && a > 1e-8;
                x = gi / (2.0 * c.ld(w[4] + i));
                break;
            }
            case R_SIN: x = gi * cos(elem(c, w[2], i)); break;
            case R_COS: x = -(gi * sin(elem(c, w[2], i))); break;
            default: {
                const double a = elem(c, w[2], i);
                x = a > 0.0 ? gi : (a < 0.0 ? -gi : 0.0);
            }
            }
            acc(c, ta, i, x, on);
        }
        break;
    }
    case R_POW: {
        const double gv = c.ld(g), a = opnd(c, w[2]), b = opnd(c, w[3]), z = c.ld(w[4]);
        const bool nz = gv != 0.0;
        acc(c, ta, 0, ((gv * b) * z) / a, nz);
        acc(c, tb, 0, (gv * z) * log(a), nz);
        break;
    }
    case R_DOT: {
        const double gv = c.ld(g);
        const bool nz = gv != 0.0;
        for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, gv * elem(c, w[3], i), nz);
        for (uint32_t i = 0; i < n; ++i) acc(c, tb, i, gv * elem(c, w[2], i), nz);
        break;
    }
    case R_MATMUL: {
        const uint32_t m = w[7] & 0xFF, k = (w[7] >> 8) & 0xFF, q = (w[7] >> 16) & 0xFF;
        double G[16], A[16], B[16];
        load_mat(c, g, m, q, G);
        bool nz = false;
#pragma unroll
        for (int i = 0; i < 16; ++i) nz = nz || G[i] != 0.0;
        if (ta != kNone) {
            load_mat(c, w[3], k, q, B);
#pragma unroll
            for (uint32_t i = 0; i < 4; ++i)
#pragma unroll
                for (uint32_t p = 0; p < 4; ++p) {
                    if (i < m && p < k) {
                        double s = G[i * 4] * B[p * 4];
#pragma unroll
                        for (uint32_t j = 1; j < 4; ++j)
                            if (j < q) s = fma(G[i * 4 + j], B[p * 4 + j], s);
                        acc(c, ta, i * k + p, s, nz);
                    }
                }
        }
        if (tb != kNone) {
            load_mat(c, w[2], m, k, A);
#pragma unroll
            for (uint32_t p = 0; p < 4; ++p)
#pragma unroll
                for (uint32_t j = 0; j < 4; ++j) {
                    if (p < k && j < q) {
                        double s = A[p] * G[j];
#pragma unroll
                        for (uint32_t i = 1; i < 4; ++i)
                            if (i < m) s = fma(A[i * 4 + p], G[i * 4 + j], s);
                        acc(c, tb, p * q + j, s, nz);
                    }
                }
        }
        break;
    }
    case R_OUTER: {
        const uint32_t m = w[7] & 0xFF, q = (w[7] >> 8) & 0xFF;
        const bool nz = any_nz(c, g, n);
        for (uint32_t i = 0; i < m; ++i) {
            double s = c.ld(g + i * q) * elem(c, w[3], 0);
            for (uint32_t j = 1; j < q; ++j) s = fma(c.ld(g + i * q + j), elem(c, w[3], j), s);
            acc(c, ta, i, s, nz);
        }
        for (uint32_t j = 0; j < q; ++j) {
            double s = c.ld(g + j) * elem(c, w[2], 0);
            for (uint32_t i = 1; i < m; ++i) s = fma(c.ld(g + i * q + j), elem(c, w[2], i), s);
            acc(c, tb, j, s, nz);
        }
        break;
    }
    case R_TRANSPOSE: {
        const uint32_t m = w[7] & 0xFF, q = (w[7] >> 8) & 0xFF;   // input m x q, g is q x m
        const bool nz = any_nz(c, g, n);
        for (uint32_t i = 0; i < m; ++i)
            for (uint32_t j = 0; j < q; ++j) acc(c, ta, i * q + j, c.ld(g + j * m + i), nz);
        break;
    }
    case R_TRACE: {
        const uint32_t sz = w[7];
        const double gv = c.ld(g);
        const bool nz = gv != 0.0;
        for (uint32_t i = 0; i < sz; ++i)
            for (uint32_t j = 0; j < sz; ++j) {
                if (i == j)
                    acc(c, ta, i * sz + j, gv, nz);
                else if (ta != kNone && (ta & kInit))
                    c.st((ta & ~kInit) + i * sz + j, 0.0);
            }
        break;
    }
    case R_INV: {
        const uint32_t sz = w[7];
        double G[16], B[16], M1[16];
        load_mat(c, g, sz, sz, G);
        load_mat(c, w[4], sz, sz, B);
        bool nz = false;
#pragma unroll
        for (int i = 0; i < 16; ++i) nz = nz || G[i] != 0.0;
        // M1 = B^T G, M2 = M1 B^T, A -= M2
#pragma unroll
        for (uint32_t i = 0; i < 2; ++i)
#pragma unroll
            for (uint32_t j = 0; j < 2; ++j) {
                double s = B[i] * G[j];
                if (sz > 1) s = fma(B[4 + i], G[4 + j], s);
                M1[i * 4 + j] = s;
            }
#pragma unroll
        for (uint32_t i = 0; i < 2; ++i)
#pragma unroll
            for (uint32_t j = 0; j < 2; ++j) {
                if (i < sz && j < sz) {
                    double s = M1[i * 4] * B[j * 4];
                    if (sz > 1) s = fma(M1[i * 4 + 1], B[j * 4 + 1], s);
                    acc(c, ta, i * sz + j, -s, nz);
                }
            }
        break;
    }
    case R_DET: case R_LOGDET: {
        const uint32_t sz = w[7];
        double A[16], Ai[16];
        load_mat(c, w[2], sz, sz, A);
        const double gv = c.ld(g);
        bool on = gv != 0.0;
        double scale;
        if (op == R_DET) {
            scale = gv * c.ld(w[4]);
        } else {
            on = on && det2(A, sz) > 1e-8;
            scale = gv;
        }
        inv2(A, sz, Ai);
#pragma unroll
        for (uint32_t i = 0; i < 2; ++i)
#pragma unroll
            for (uint32_t j = 0; j < 2; ++j)
                if (i < sz && j < sz) acc(c, ta, i * sz + j, scale * Ai[j * 4 + i], on);
        break;
    }
    case R_PACK: {
        const bool nz = any_nz(c, g, n);
        for (uint32_t i = 0; i < n; ++i) acc(c, C::aux_word(aux, w[7] + i), 0, c.ld(g + i), nz);
        break;
    }
    case R_INDEX: {
        const double gv = c.ld(g);
        const bool nz = gv != 0.0;
        if (ta != kNone && (ta & kInit)) {
            for (uint32_t i = 0; i < n; ++i)
                if (i != w[7]) c.st((ta & ~kInit) + i, 0.0);
        }
        acc(c, ta, w[7], gv, nz);
        break;
    }
    case R_SELECT: {
        const bool p = opnd(c, w[2]) < opnd(c, w[3]);
        const bool nz = any_nz(c, g, n);
        for (uint32_t i = 0; i < n; ++i) acc(c, ta, i, c.ld(g + i), nz && p);
        for (uint32_t i = 0; i < n; ++i) acc(c, tb, i, c.ld(g + i), nz && !p);
        break;
    }
    default:
        break;
    }
}


// adjoint update of a scalar target (see acc); never kNone here (the
// scheduler points unused targets at a sink register), so no branch
template <class C>
NDVM_HD void acc1(const C &c, uint32_t tw, double x, bool on) {
    const uint32_t r = tw & ~kInit;
    const double old = c.ld_raw(r);   // may be unset when the first contribution stores
    const double base = (tw & kInit) ? 0.0 : old;
    c.st(r, on ? base + x : base);
}

// Scalar handlers without any data-dependent control flow inside: kept in a
// switch of their own so the compiler can leave that region's uniform
// branches unstructured (a direct jump back to the dispatch).
constexpr uint32_t kHotMask =
    (1u << (S_ADD - S_ADD)) | (1u << (S_SUB - S_ADD)) | (1u << (S_MUL - S_ADD)) | (1u << (S_DIV - S_ADD)) |
    (1u << (S_NEG - S_ADD)) | (1u << (S_ABS - S_ADD)) | (1u << (S_SELECT - S_ADD)) | (1u << (F2 - S_ADD)) | (1u << (R2 - S_ADD)) |
    (1u << (SR_ADD - S_ADD)) | (1u << (SR_SUB - S_ADD)) | (1u << (SR_MUL - S_ADD)) |
    (1u << (SR_DIV - S_ADD)) | (1u << (SR_NEG - S_ADD)) | (1u << (SR_EXP - S_ADD)) |
    (1u << (SR_LOG - S_ADD)) | (1u << (SR_SQRT - S_ADD)) | (1u << (SR_ABS - S_ADD)) |
    (1u << (SR_SELECT - S_ADD));

// scalar binary op selected by a wave-uniform sub-op code
NDVM_HD double binop(uint32_t sub, double a, double b) {
    switch (sub) {
    case 0: return a + b;
    case 1: return a - b;
    case 2: return a * b;
    default: return a / b;
    }
}

// contributions of one scalar binary adjoint rule (sub-op as in binop)
template <class C>
NDVM_HD void rev_binop(const C &c, uint32_t sub, uint32_t wg, uint32_t wa, uint32_t wb, uint32_t wz,
                       uint32_t ta, uint32_t tb) {
    const double g = c.ld(wg);
    const bool nz = g != 0.0;
    switch (sub) {
    case 0:
        acc1(c, ta, g, nz);
        acc1(c, tb, g, nz);
        return;
    case 1:
        acc1(c, ta, g, nz);
        acc1(c, tb, -g, nz);
        return;
    case 2: {
        const double a = c.ld(wa), b = c.ld(wb);
        acc1(c, ta, g * b, nz);
        acc1(c, tb, g * a, nz);
        return;
    }
    default: {
        const double b = c.ld(wb), z = c.ld(wz);
        acc1(c, ta, g / b, nz);
        acc1(c, tb, -((g * z) / b), nz);
        return;
    }
    }
}

// a 16-bit target field as a target word
NDVM_HD uint32_t t16(uint32_t f) { return (f & 0x7FFFu) | ((f & 0x8000u) << 16); }

template <class C>
NDVM_HD void exec_hot(const C &c, const uint32_t *w, uint32_t op) {
    switch (op) {
    case R2: {
        const uint32_t h = C::uni(w[0]);
        rev_binop(c, (h >> 8) & 15u, w[1] & 0xFFFFu, w[1] >> 16, w[2] & 0xFFFFu, w[2] >> 16,
                  t16(w[3] & 0xFFFFu), t16(w[3] >> 16));
        rev_binop(c, (h >> 12) & 15u, w[4] & 0xFFFFu, w[4] >> 16, w[5] & 0xFFFFu, w[5] >> 16,
                  t16(w[6] & 0xFFFFu), t16(w[6] >> 16));
        return;
    }
    case F2: {
        const uint32_t h = C::uni(w[0]);
        const double a1 = c.ld(w[2]), b1 = c.ld(w[3]), a2 = c.ld(w[5]), b2 = c.ld(w[6]);
        c.st(w[1], binop((h >> 8) & 15u, a1, b1));
        c.st(w[4], binop((h >> 12) & 15u, a2, b2));
        return;
    }
    case S_ADD: c.st(w[1], c.ld(w[2]) + c.ld(w[3])); return;
    case S_SUB: c.st(w[1], c.ld(w[2]) - c.ld(w[3])); return;
    case S_MUL: c.st(w[1], c.ld(w[2]) * c.ld(w[3])); return;
    case S_DIV: c.st(w[1], c.ld(w[2]) / c.ld(w[3])); return;
    case S_NEG: c.st(w[1], -c.ld(w[2])); return;
    case S_ABS: c.st(w[1], fabs(c.ld(w[2]))); return;
    case S_SELECT: {
        const bool p = c.ld(w[2]) < c.ld(w[3]);
        const double x = c.ld(w[4]), y = c.ld(w[5]);
        c.st(w[1], p ? x : y);
        return;
    }
    case SR_ADD: {
        const double g = c.ld(w[1]);
        const bool nz = g != 0.0;
        acc1(c, w[5], g, nz);
        acc1(c, w[6], g, nz);
        return;
    }
    case SR_SUB: {
        const double g = c.ld(w[1]);
        const bool nz = g != 0.0;
        acc1(c, w[5], g, nz);
        acc1(c, w[6], -g, nz);
        return;
    }
    case SR_MUL: {
        const double g = c.ld(w[1]), a = c.ld(w[2]), b = c.ld(w[3]);
        const bool nz = g != 0.0;
        acc1(c, w[5], g * b, nz);
        acc1(c, w[6], g * a, nz);
        return;
    }
    case SR_DIV: {
        const double g = c.ld(w[1]), b = c.ld(w[3]), z = c.ld(w[4]);
        const bool nz = g != 0.0;
        acc1(c, w[5], g / b, nz);
        acc1(c, w[6], -((g * z) / b), nz);
        return;
    }
    case SR_NEG: {
        const double g = c.ld(w[1]);
        acc1(c, w[5], -g, g != 0.0);
        return;
    }
    case SR_EXP: {
        const double g = c.ld(w[1]);
        acc1(c, w[5], g * c.ld(w[4]), g != 0.0);
        return;
    }
    case SR_LOG: {
        const double g = c.ld(w[1]), a = c.ld(w[2]);
        acc1(c, w[5], g / a, g != 0.0 && a > 1e-8);
        return;
    }
    case SR_SQRT: {
        const double g = c.ld(w[1]), a = c.ld(w[2]);
        acc1(c, w[5], g / (2.0 * c.ld(w[4])), g != 0.0 && a > 1e-8);
        return;
    }
    case SR_ABS: {
        const double g = c.ld(w[1]), a = c.ld(w[2]);
        acc1(c, w[5], a > 0.0 ? g : (a < 0.0 ? -g : 0.0), g != 0.0);
        return;
    }
    case SR_SELECT: {
        const double g = c.ld(w[1]);
        const bool nz = g != 0.0;
        const bool p = c.ld(w[2]) < c.ld(w[3]);
        acc1(c, w[5], g, nz && p);
        acc1(c, w[6], g, nz && !p);
        return;
    }
    default:
        return;
    }
}

// remaining scalar fast paths (transcendentals, whose library code branches
// on the argument)
template <class C>
NDVM_HD void exec_scalar(const C &c, const uint32_t *w) {
    const uint32_t op = w[0] & 0xFF;
    switch (op) {
    case S_EXP: c.st(w[1], exp(c.ld(w[2]))); return;
    case S_LOG: c.st(w[1], log(clampv(c.ld(w[2])))); return;
    case S_SQRT: c.st(w[1], sqrt(clampv(c.ld(w[2])))); return;
    case S_SIN: c.st(w[1], sin(c.ld(w[2]))); return;
    case S_COS: c.st(w[1], cos(c.ld(w[2]))); return;
    case SR_SIN: {
        const double g = c.ld(w[1]);
        acc1(c, w[5], g * cos(c.ld(w[2])), g != 0.0);
        return;
    }
    case SR_COS: {
        const double g = c.ld(w[1]);
        acc1(c, w[5], -(g * sin(c.ld(w[2]))), g != 0.0);
        return;
    }
    default:
        return;
    }
}

// Execute one instruction; false at END.  `wv` are the instruction words as
// loaded (on the GPU: vector registers holding the same value in every
// lane); the hot scalar handlers use them directly as LDS addresses, all
// other paths first make every word an explicit scalar.
template <class C>
NDVM_HD bool step(const C &c, const uint32_t *wv, const uint32_t *aux) {
    const uint32_t op = C::uni(wv[0]) & 0xFF;
    if (op >= S_ADD && ((kHotMask >> (op - S_ADD)) & 1u)) {
        exec_hot(c, wv, op);
        return true;
    }
    uint32_t w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = C::uni(wv[i]);
    if (op >= S_ADD) {
        exec_scalar(c, w);
        return true;
    }
    if (op >= R_ADD) {
        exec_rev(c, aux, w);
        return true;
    }
    if (op >= F_ADD) {
        exec_fwd(c, aux, w);
        return true;
    }
    const uint32_t n = (w[0] >> 16) & 0xFF;
    switch (op) {
    case END:
        return false;
    case LDPARAM:
        c.st(w[1], c.param(w[7]));
        break;
    case ST_LOSS:
        c.store_loss(c.ld(w[2]));
        break;
    case CKPT_ST:
        for (uint32_t i = 0; i < n; ++i) c.ckpt_st(w[7] + i, c.ld(w[2] + i));
        break;
    case CKPT_LD:
        for (uint32_t i = 0; i < n; ++i) c.st(w[1] + i, c.ckpt_ld(w[7] + i));
        break;
    case ZERO:
        for (uint32_t i = 0; i < n; ++i) c.st(w[1] + i, 0.0);
        break;
    case SEED:
        acc(c, w[5], 0, 1.0, true);
        break;
    case ST_GRAD:
        c.store_grad(w[7], c.ld(w[2]));
        break;
    case LDOBS:
        c.st(w[1], c.obsv(w[7]));
        break;
    case LDCONST:
        for (uint32_t i = 0; i < n; ++i) c.st(w[1] + i, c.konst(w[7] + i));
        break;
    default:
        return false;
    }
    return true;
}

// Execute a device program from `pc` until END.  Instructions are fetched two
// ahead (programs end with padding instructions of END so the look-ahead stays
// inside the program).
template <class C>
NDVM_HD void run(const C &c, const uint32_t *pc, const uint32_t *aux) {
    typename C::Fetch f0 = C::prefetch(pc), f1 = C::prefetch(pc + kWords);
    for (;; pc += kWords) {
        typename C::Fetch f2 = C::prefetch(pc + 2 * kWords);
        uint32_t wv[8];
        C::decode(f0, wv);
        if (!step(c, wv, aux)) return;
        f0 = f1;
        f1 = f2;
    }
}

}  // namespace replay
}  // namespace ndvm
