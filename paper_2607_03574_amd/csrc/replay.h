// Instruction handlers of the device program, shared by the GPU replay
// kernel and the host-side emulator used to check the scheduler.
//
// A context type C supplies the lane's register file and memory:
//   double ld(uint32_t r) const;  void st(uint32_t r, double v) const;
//   double ld_raw(uint32_t r) const;   (a read whose value may be discarded)
//   double konst(uint32_t i) const;  double obsv(uint32_t i) const;  (uniform loads)
//   static uint32_t uni(uint32_t x);          (wave-uniform value)
//   static bool all(bool b);                  (b holds in every lane of the wave)
//   double ldh(uint32_t word, int hi) const;  void sth(uint32_t word, int hi, double v) const;
//   double ldh_raw(uint32_t word, int hi) const;
//        (the register named by the low (hi = 0) or high half of `word`)
//   Chunk load_chunk(const uint32_t *p) const;   (kChunkInstr instructions)
//   static Words instr(const Chunk&, uint32_t i);  (instruction i; Words[k] = word k, uniform)
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

// ---- small-matrix fast paths: shapes known at compile time, so every loop
// unrolls, element offsets become immediate LDS offsets and no per-element
// branch remains.  Same arithmetic as the generic handlers: ascending fma
// chains whose first term is a plain product.

// adjoint update of register r (first contribution when `init`), as acc
template <class C>
NDVM_HD void accv(const C &c, uint32_t r, bool init, double x, bool on) {
    const double old = c.ld_raw(r);   // may be unset on a first contribution
    const double b = init ? 0.0 : old;
    c.st(r, on ? b + x : b);
}

// Adjoint update of the E registers r.. with contributions T, gated per lane
// on `nz`, as accv element by element.  `init` is uniform, so it selects a
// code path instead of a value; when every lane of the wave has nz the gate
// is the identity and its selects are skipped.
template <int E, class C>
NDVM_HD void acc_block(const C &c, uint32_t r, bool init, const double (&T)[E], bool nz) {
    const bool all = C::all(nz);
    if (init) {
        if (all) {
#pragma unroll
            for (int e = 0; e < E; ++e) c.st(r + e, 0.0 + T[e]);
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e) c.st(r + e, nz ? 0.0 + T[e] : 0.0);
        }
        return;
    }
    double old[E];
#pragma unroll
    for (int e = 0; e < E; ++e) old[e] = c.ld(r + e);
    if (all) {
#pragma unroll
        for (int e = 0; e < E; ++e) c.st(r + e, old[e] + T[e]);
    } else {
#pragma unroll
        for (int e = 0; e < E; ++e) c.st(r + e, nz ? old[e] + T[e] : old[e]);
    }
}

template <int M, int K, int N, class C>
NDVM_HD void mm_fwd(const C &c, uint32_t d, uint32_t a, uint32_t b) {
    double A[M * K], B[K * N];
#pragma unroll
    for (int i = 0; i < M * K; ++i) A[i] = c.ld(a + i);
#pragma unroll
    for (int i = 0; i < K * N; ++i) B[i] = c.ld(b + i);
#pragma unroll
    for (int i = 0; i < M; ++i)
#pragma unroll
        for (int j = 0; j < N; ++j) {
            double s = A[i * K] * B[j];
#pragma unroll
            for (int p = 1; p < K; ++p) s = fma(A[i * K + p], B[p * N + j], s);
            c.st(d + i * N + j, s);
        }
}

// Z = A B with adjoint G: A += G B^T, B += A^T G, gated on any G != 0
template <int M, int K, int N, class C>
NDVM_HD void mm_rev(const C &c, uint32_t g, uint32_t a, uint32_t b, uint32_t ta, uint32_t tb) {
    double G[M * N];
    bool nz = false;
#pragma unroll
    for (int i = 0; i < M * N; ++i) {
        G[i] = c.ld(g + i);
        nz = nz || G[i] != 0.0;
    }
    if (ta != kNone) {
        const uint32_t r = ta & ~kInit;
        const bool init = (ta & kInit) != 0;
        double B[K * N], T[M * K];
#pragma unroll
        for (int i = 0; i < K * N; ++i) B[i] = c.ld(b + i);
#pragma unroll
        for (int i = 0; i < M; ++i)
#pragma unroll
            for (int q = 0; q < K; ++q) {
                double s = G[i * N] * B[q * N];
#pragma unroll
                for (int j = 1; j < N; ++j) s = fma(G[i * N + j], B[q * N + j], s);
                T[i * K + q] = s;
            }
        acc_block<M * K>(c, r, init, T, nz);
    }
    if (tb != kNone) {
        const uint32_t r = tb & ~kInit;
        const bool init = (tb & kInit) != 0;
        double A[M * K], T[K * N];
#pragma unroll
        for (int i = 0; i < M * K; ++i) A[i] = c.ld(a + i);
#pragma unroll
        for (int q = 0; q < K; ++q)
#pragma unroll
            for (int j = 0; j < N; ++j) {
                double s = A[q] * G[j];
#pragma unroll
                for (int i = 1; i < M; ++i) s = fma(A[i * K + q], G[i * N + j], s);
                T[q * N + j] = s;
            }
        acc_block<K * N>(c, r, init, T, nz);
    }
}

#define NDVM_MM_SHAPES(X) \
    X(1, 1, 1) X(1, 1, 2) X(1, 1, 4) X(1, 2, 1) X(1, 2, 2) X(1, 2, 4) X(1, 4, 1) X(1, 4, 2) X(1, 4, 4) \
    X(2, 1, 1) X(2, 1, 2) X(2, 1, 4) X(2, 2, 1) X(2, 2, 2) X(2, 2, 4) X(2, 4, 1) X(2, 4, 2) X(2, 4, 4) \
    X(4, 1, 1) X(4, 1, 2) X(4, 1, 4) X(4, 2, 1) X(4, 2, 2) X(4, 2, 4) X(4, 4, 1) X(4, 4, 2) X(4, 4, 4)

// shapes with m, k, n in {1, 2, 4}; false for the generic handler
template <class C, class W>
NDVM_HD bool mm_fwd_fast(const C &c, const W &w) {
    switch (w[7] & 0xFFFFFFu) {
#define NDVM_X(m, k, n) \
    case (m) | ((k) << 8) | ((n) << 16): mm_fwd<m, k, n>(c, w[1], w[2], w[3]); return true;
        NDVM_MM_SHAPES(NDVM_X)
#undef NDVM_X
    }
    return false;
}
template <class C, class W>
NDVM_HD bool mm_rev_fast(const C &c, const W &w) {
    switch (w[7] & 0xFFFFFFu) {
#define NDVM_X(m, k, n) \
    case (m) | ((k) << 8) | ((n) << 16): mm_rev<m, k, n>(c, w[1], w[2], w[3], w[5], w[6]); return true;
        NDVM_MM_SHAPES(NDVM_X)
#undef NDVM_X
    }
    return false;
}

// elementwise binary ops of two equal-shape operands, N elements
template <int N, class C>
NDVM_HD void ew_fwd(const C &c, uint32_t op, uint32_t d, uint32_t a, uint32_t b) {
    double x[N], y[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        x[i] = c.ld(a + i);
        y[i] = c.ld(b + i);
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const double z = op == F_ADD ? x[i] + y[i] : op == F_SUB ? x[i] - y[i] : op == F_MUL ? x[i] * y[i]
                                                                                              : x[i] / y[i];
        c.st(d + i, z);
    }
}
// adjoints of an elementwise sum or difference, N elements
template <int N, class C>
NDVM_HD void ew_rev_addsub(const C &c, bool sub, uint32_t g, uint32_t ta, uint32_t tb) {
    double G[N];
    bool nz = false;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        G[i] = c.ld(g + i);
        nz = nz || G[i] != 0.0;
    }
    if (ta != kNone) acc_block<N>(c, ta & ~kInit, (ta & kInit) != 0, G, nz);
    if (tb != kNone) {
        double H[N];
#pragma unroll
        for (int i = 0; i < N; ++i) H[i] = sub ? -G[i] : G[i];
        acc_block<N>(c, tb & ~kInit, (tb & kInit) != 0, H, nz);
    }
}

template <class C, class W>
NDVM_HD bool ew_fwd_fast(const C &c, const W &w, uint32_t op) {
    const uint32_t w0 = w[0];
    if (((w0 >> 8) & 0xFF) != MODE_SAME) return false;
    switch ((w0 >> 16) & 0xFF) {
    case 2: ew_fwd<2>(c, op, w[1], w[2], w[3]); return true;
    case 4: ew_fwd<4>(c, op, w[1], w[2], w[3]); return true;
    case 16: ew_fwd<16>(c, op, w[1], w[2], w[3]); return true;
    }
    return false;
}
template <class C, class W>
NDVM_HD bool ew_rev_fast(const C &c, const W &w, uint32_t op) {
    switch ((w[0] >> 16) & 0xFF) {
    case 2: ew_rev_addsub<2>(c, op == R_SUB, w[1], w[5], w[6]); return true;
    case 4: ew_rev_addsub<4>(c, op == R_SUB, w[1], w[5], w[6]); return true;
    case 16: ew_rev_addsub<16>(c, op == R_SUB, w[1], w[5], w[6]); return true;
    }
    return false;
}

// checkpoint rows to registers and back, N elements: every load is issued
// before the first store
template <int N, class C>
NDVM_HD void ckpt_load(const C &c, uint32_t d, uint32_t row) {
    double v[N];
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = c.ckpt_ld(row + i);
#pragma unroll
    for (int i = 0; i < N; ++i) c.st(d + i, v[i]);
}
template <int N, class C>
NDVM_HD void ckpt_store(const C &c, uint32_t src, uint32_t row) {
    double v[N];
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = c.ld(src + i);
#pragma unroll
    for (int i = 0; i < N; ++i) c.ckpt_st(row + i, v[i]);
}
template <class C, class W>
NDVM_HD bool ckpt_fast(const C &c, const W &w, bool load) {
    const uint32_t n = (w[0] >> 16) & 0xFF;
    switch (n) {
    case 1: load ? ckpt_load<1>(c, w[1], w[7]) : ckpt_store<1>(c, w[2], w[7]); return true;
    case 2: load ? ckpt_load<2>(c, w[1], w[7]) : ckpt_store<2>(c, w[2], w[7]); return true;
    case 4: load ? ckpt_load<4>(c, w[1], w[7]) : ckpt_store<4>(c, w[2], w[7]); return true;
    case 16: load ? ckpt_load<16>(c, w[1], w[7]) : ckpt_store<16>(c, w[2], w[7]); return true;
    }
    return false;
}

// Register named by 16-bit field i of a bundle instruction: word and half.
// The context loads and stores through (word, half) so the GPU can form the
// address from the scalar word in one instruction.
#define NDVM_FW(i) ((i) == 14 ? w[0] : w[1 + ((i) >> 1)])
#define NDVM_FH(i) ((i) == 14 ? 1 : ((i) & 1))

// d = fma(x, y, w) for N independent ops; all operands are read before any
// result is written (the scheduler never bundles an op with one it reads)
template <int N, class C, class W>
NDVM_HD void fma_bundle(const C &c, const W &w) {
    double x[N], y[N], z[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
        x[k] = c.ldh(NDVM_FW(4 * k + 1), NDVM_FH(4 * k + 1));
        y[k] = c.ldh(NDVM_FW(4 * k + 2), NDVM_FH(4 * k + 2));
        z[k] = c.ldh(NDVM_FW(4 * k + 3), NDVM_FH(4 * k + 3));
    }
#pragma unroll
    for (int k = 0; k < N; ++k) c.sth(NDVM_FW(4 * k), NDVM_FH(4 * k), fma(x[k], y[k], z[k]));
}

template <int N, class C, class W>
NDVM_HD void div_bundle(const C &c, const W &w) {
    double a[N], b[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
        a[k] = c.ldh(NDVM_FW(3 * k + 1), NDVM_FH(3 * k + 1));
        b[k] = c.ldh(NDVM_FW(3 * k + 2), NDVM_FH(3 * k + 2));
    }
#pragma unroll
    for (int k = 0; k < N; ++k) c.sth(NDVM_FW(3 * k), NDVM_FH(3 * k), a[k] / b[k]);
}

// adjoint rules of N bundled ops (kDiv: division rule, else linear).  Every
// g and operand is read first.  With distinct targets (!kSeq) every target is
// read before any is written; otherwise each target is read just before it is
// written, after the earlier rules' updates (LDS accesses of a wave are
// performed in order).
template <int N, bool kDiv, bool kSeq, class C, class W>
NDVM_HD void adj_bundle(const C &c, const W &w) {
    const uint32_t w0 = w[0];
    double g[N], p[N], q[N], xa[N], xb[N], oa[N], ob[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
        g[k] = c.ldh(NDVM_FW(5 * k), NDVM_FH(5 * k));
        p[k] = c.ldh(NDVM_FW(5 * k + 1), NDVM_FH(5 * k + 1));
        q[k] = c.ldh(NDVM_FW(5 * k + 2), NDVM_FH(5 * k + 2));
        if (!kSeq) {   // may be unset on a first contribution
            oa[k] = c.ldh_raw(NDVM_FW(5 * k + 3), NDVM_FH(5 * k + 3));
            ob[k] = c.ldh_raw(NDVM_FW(5 * k + 4), NDVM_FH(5 * k + 4));
        }
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
        if (kDiv) {
            xa[k] = g[k] / p[k];
            xb[k] = -((g[k] * q[k]) / p[k]);
        } else {
            xa[k] = g[k] * p[k];
            xb[k] = g[k] * q[k];
        }
    }
#pragma unroll
    for (int k = 0; k < N; ++k) {
        const bool nz = g[k] != 0.0;
        if (kSeq) oa[k] = c.ldh_raw(NDVM_FW(5 * k + 3), NDVM_FH(5 * k + 3));
        const double ba = (w0 >> (8 + 2 * k)) & 1u ? 0.0 : oa[k];
        c.sth(NDVM_FW(5 * k + 3), NDVM_FH(5 * k + 3), nz ? ba + xa[k] : ba);
        if (kSeq) ob[k] = c.ldh_raw(NDVM_FW(5 * k + 4), NDVM_FH(5 * k + 4));
        const double bb = (w0 >> (9 + 2 * k)) & 1u ? 0.0 : ob[k];
        c.sth(NDVM_FW(5 * k + 4), NDVM_FH(5 * k + 4), nz ? bb + xb[k] : bb);
    }
}
#undef NDVM_FW
#undef NDVM_FH

// N observation loads: word k + 1 = destination | observation index << 16;
// every (scalar) load is issued before the first store
template <int N, class C, class W>
NDVM_HD void obs_bundle(const C &c, const W &w) {
    double v[N];
#pragma unroll
    for (int k = 0; k < N; ++k) v[k] = c.obsv(w[1 + k] >> 16);
#pragma unroll
    for (int k = 0; k < N; ++k) c.sth(w[1 + k], 0, v[k]);
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

// Everything but END and the scalar/bundle fast paths: generic element
// loops, scalar transcendentals, parameter, constant, observation, checkpoint
// and gradient traffic.
template <class C>
NDVM_HD void exec_cold(const C &c, const uint32_t *w, uint32_t op, const uint32_t *aux) {
    if (op >= S_ADD) {
        exec_scalar(c, w);
        return;
    }
    if (op >= R_ADD) {
        exec_rev(c, aux, w);
        return;
    }
    if (op >= F_ADD) {
        exec_fwd(c, aux, w);
        return;
    }
    const uint32_t n = (w[0] >> 16) & 0xFF;
    switch (op) {
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
        break;
    }
}

// Execute a device program until END.  One flat switch over the opcodes in
// a loop without exits, so every handler jumps straight back to the fetch.  `wv[k]` is word k of the
// current instruction (wave-uniform); handlers read only the words they use.
// The chunk after the current one is loaded when the current one starts, so
// it has a whole chunk's worth of instructions to arrive (programs are padded
// so this read-ahead stays inside the program).
// all eight words of an instruction as an array
struct Words8 {
    uint32_t v[8];
};
template <class W>
NDVM_HD Words8 words8(const W &w) {
    Words8 r;
#pragma unroll
    for (int k = 0; k < 8; ++k) r.v[k] = w[k];
    return r;
}

// Run `body` (which reads the instruction through `w`) for instruction i and,
// while its repeat bit is set, for the next instructions of the chunk (same
// opcode), without going back through the dispatch; leaves i on the last one.
#define NDVM_RUN(body)                             \
    for (auto w = C::instr(cur, i);;) {            \
        body;                                      \
        if (!(w[0] & kRepeat)) break;              \
        w = C::instr(cur, ++i);                    \
    }

template <class C>
NDVM_HD void run(const C &c, const uint32_t *prog, const uint32_t *aux) {
    typename C::Chunk cur = c.load_chunk(prog), nxt = c.load_chunk(prog + kChunkWords);
    for (const uint32_t *ahead = prog + 2 * kChunkWords;; ahead += kChunkWords) {
        // END only ever opens a chunk; the chunk registers change only below,
        // outside the per-instruction loop, which has no exit of its own
        if ((C::instr(cur, 0)[0] & 0xFF) == END) return;
        for (uint32_t i = 0; i < kChunkInstr; ++i) {
            const auto w = C::instr(cur, i);
            const uint32_t op = w[0] & 0xFF;
            switch (op) {
            case END: case NOP: break;
            case FB1: NDVM_RUN((fma_bundle<1>(c, w))) break;
            case FB2: NDVM_RUN((fma_bundle<2>(c, w))) break;
            case FB3: NDVM_RUN((fma_bundle<3>(c, w))) break;
            case DB1: NDVM_RUN((div_bundle<1>(c, w))) break;
            case DB2: NDVM_RUN((div_bundle<2>(c, w))) break;
            case DB3: NDVM_RUN((div_bundle<3>(c, w))) break;
            case LB1: NDVM_RUN((adj_bundle<1, false, false>(c, w))) break;
            case LB2: NDVM_RUN((adj_bundle<2, false, false>(c, w))) break;
            case LB3: NDVM_RUN((adj_bundle<3, false, false>(c, w))) break;
            case RDB1: NDVM_RUN((adj_bundle<1, true, false>(c, w))) break;
            case RDB2: NDVM_RUN((adj_bundle<2, true, false>(c, w))) break;
            case RDB3: NDVM_RUN((adj_bundle<3, true, false>(c, w))) break;
            case LBS1: NDVM_RUN((adj_bundle<1, false, true>(c, w))) break;
            case LBS2: NDVM_RUN((adj_bundle<2, false, true>(c, w))) break;
            case LBS3: NDVM_RUN((adj_bundle<3, false, true>(c, w))) break;
            case RDBS1: NDVM_RUN((adj_bundle<1, true, true>(c, w))) break;
            case RDBS2: NDVM_RUN((adj_bundle<2, true, true>(c, w))) break;
            case RDBS3: NDVM_RUN((adj_bundle<3, true, true>(c, w))) break;
            case OB2: NDVM_RUN((obs_bundle<2>(c, w))) break;
            case OB3: NDVM_RUN((obs_bundle<3>(c, w))) break;
            case OB4: NDVM_RUN((obs_bundle<4>(c, w))) break;
            case S_ADD: c.st(w[1], c.ld(w[2]) + c.ld(w[3])); break;
            case S_SUB: c.st(w[1], c.ld(w[2]) - c.ld(w[3])); break;
            case S_MUL: c.st(w[1], c.ld(w[2]) * c.ld(w[3])); break;
            case S_DIV: c.st(w[1], c.ld(w[2]) / c.ld(w[3])); break;
            case S_NEG: c.st(w[1], -c.ld(w[2])); break;
            case S_ABS: c.st(w[1], fabs(c.ld(w[2]))); break;
            case S_SELECT: {
                const bool p = c.ld(w[2]) < c.ld(w[3]);
                const double x = c.ld(w[4]), y = c.ld(w[5]);
                c.st(w[1], p ? x : y);
                break;
            }
            case SR_ADD: {
                const double g = c.ld(w[1]);
                const bool nz = g != 0.0;
                acc1(c, w[5], g, nz);
                acc1(c, w[6], g, nz);
                break;
            }
            case SR_SUB: {
                const double g = c.ld(w[1]);
                const bool nz = g != 0.0;
                acc1(c, w[5], g, nz);
                acc1(c, w[6], -g, nz);
                break;
            }
            case SR_MUL: {
                const double g = c.ld(w[1]), a = c.ld(w[2]), b = c.ld(w[3]);
                const bool nz = g != 0.0;
                acc1(c, w[5], g * b, nz);
                acc1(c, w[6], g * a, nz);
                break;
            }
            case SR_DIV: {
                const double g = c.ld(w[1]), b = c.ld(w[3]), z = c.ld(w[4]);
                const bool nz = g != 0.0;
                acc1(c, w[5], g / b, nz);
                acc1(c, w[6], -((g * z) / b), nz);
                break;
            }
            case SR_NEG: {
                const double g = c.ld(w[1]);
                acc1(c, w[5], -g, g != 0.0);
                break;
            }
            case SR_EXP: {
                const double g = c.ld(w[1]);
                acc1(c, w[5], g * c.ld(w[4]), g != 0.0);
                break;
            }
            case SR_LOG: {
                const double g = c.ld(w[1]), a = c.ld(w[2]);
                acc1(c, w[5], g / a, g != 0.0 && a > 1e-8);
                break;
            }
            case SR_SQRT: {
                const double g = c.ld(w[1]), a = c.ld(w[2]);
                acc1(c, w[5], g / (2.0 * c.ld(w[4])), g != 0.0 && a > 1e-8);
                break;
            }
            case SR_ABS: {
                const double g = c.ld(w[1]), a = c.ld(w[2]);
                acc1(c, w[5], a > 0.0 ? g : (a < 0.0 ? -g : 0.0), g != 0.0);
                break;
            }
            case SR_SELECT: {
                const double g = c.ld(w[1]);
                const bool nz = g != 0.0;
                const bool p = c.ld(w[2]) < c.ld(w[3]);
                acc1(c, w[5], g, nz && p);
                acc1(c, w[6], g, nz && !p);
                break;
            }
            case F_MATMUL:
                NDVM_RUN(if (!mm_fwd_fast(c, w)) exec_fwd(c, aux, words8(w).v))
                break;
            case R_MATMUL:
                NDVM_RUN(if (!mm_rev_fast(c, w)) exec_rev(c, aux, words8(w).v))
                break;
            case F_ADD: case F_SUB: case F_MUL: case F_DIV:
                if (!ew_fwd_fast(c, w, op)) goto cold;
                break;
            case R_ADD: case R_SUB:
                if (!ew_rev_fast(c, w, op)) goto cold;
                break;
            case CKPT_LD:
                if (!ckpt_fast(c, w, true)) goto cold;
                break;
            case CKPT_ST:
                if (!ckpt_fast(c, w, false)) goto cold;
                break;
            case LDOBS: c.st(w[1], c.obsv(w[7])); break;
            default:
            cold: {
                uint32_t wc[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) wc[k] = w[k];
                exec_cold(c, wc, op, aux);
                break;
            }
            }
        }
        cur = nxt;
        nxt = c.load_chunk(ahead);
    }
}
#undef NDVM_RUN

}  // namespace replay
}  // namespace ndvm
