// Device walker kernel: the structural walk of a stack-bytecode program on
// the GPU, one wave per 64 lanes of one program (definitions and layout in
// walk.h).
//
// Control is the same for every lane of a wave: program counter, operand
// stack (node numbers), locals, loop counters and branch frames live once
// per wave in LDS and are read back as wave-uniform values.  Numbers are
// per lane: node k's values are a coalesced row of 64 doubles in the wave's
// HBM slot.  A numeric IFLT takes one ballot: each arm runs under the mask
// of the lanes that take it, an arm no lane takes is not walked at all, and
// when both arms ran their differing stack positions and locals become MERGE
// nodes (Section 6, lane masking).  The reverse sweep visits the recorded
// nodes from last to first and applies the adjoint rules of Appendix C,
// table tab:adjoints, per lane, gated on a nonzero incoming adjoint; an
// adjoint row is written in full by its first contribution (zero where the
// rule does not apply), so no row is cleared beforehand, and a node no rule
// reached is skipped without a read.
#include <hip/hip_runtime.h>

#include <cmath>

#include "common.h"
#include "walk.h"

namespace ndvm {
namespace {

using walk::Args;
using walk::Node;
using walk::ProgDesc;

constexpr uint32_t kUnset = 0xFFFFFFFFu;

__device__ __forceinline__ uint32_t uni(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint64_t uni64(uint64_t v) {
    return uint64_t(uni(uint32_t(v))) | uint64_t(uni(uint32_t(v >> 32))) << 32;
}

__device__ __forceinline__ double clampv(double x) { return x < 1e-8 ? 1e-8 : x; }

__device__ __forceinline__ bool is_binary(uint32_t op) {
    return op == bc::ADD || op == bc::SUB || op == bc::MUL || op == bc::DIV || op == bc::POW;
}

// forward value of a scalar word
__device__ __forceinline__ double forward(uint32_t op, double x, double y) {
    switch (op) {
    case bc::ADD: return x + y;
    case bc::SUB: return x - y;
    case bc::MUL: return x * y;
    case bc::DIV: return x / y;
    case bc::NEG: return -x;
    case bc::EXP: return exp(x);
    case bc::LOG: return log(clampv(x));
    case bc::SQRT: return sqrt(clampv(x));
    case bc::SIN: return sin(x);
    case bc::COS: return cos(x);
    case bc::ABS: return fabs(x);
    default: return pow(x, y);   // POW
    }
}

// operand stack words a bytecode word pops and pushes
__device__ __forceinline__ void stack_effect(uint32_t op, uint32_t *pops, uint32_t *pushes) {
    switch (op) {
    case bc::PUSH: case bc::OBS: case bc::PARAM: case bc::LOADL: *pops = 0; *pushes = 1; return;
    case bc::STOREL: case bc::DROP: *pops = 1; *pushes = 0; return;
    case bc::DUP: *pops = 1; *pushes = 2; return;
    case bc::OVER: *pops = 2; *pushes = 3; return;
    case bc::SWAP: *pops = 2; *pushes = 2; return;
    case bc::IFLT: *pops = 2; *pushes = 0; return;
    case bc::HALT: case bc::LOOP: case bc::ENDLOOP: case bc::ELSE: case bc::ENDIF: *pops = 0; *pushes = 0; return;
    default: *pops = is_binary(op) ? 2 : 1; *pushes = 1; return;
    }
}

struct Wave {
    uint32_t lane;
    uint32_t *stk, *loc, *lps, *frm, *flg;
    uint32_t snap, fsz, depth;
    double *V, *G;
    Node *E;

    // two flag bits per node in LDS: bit 0 leaf, bit 1 adjoint row written
    __device__ __forceinline__ uint32_t flags(uint32_t k) const { return uni(flg[k >> 4]) >> ((k & 15) * 2) & 3u; }
    __device__ __forceinline__ void set_flag(uint32_t k, uint32_t bit) const {
        const uint32_t w = uni(flg[k >> 4]);
        flg[k >> 4] = w | bit << ((k & 15) * 2);
    }
    __device__ __forceinline__ double &v(uint32_t k) const { return V[uint64_t(k) * 64 + lane]; }
    __device__ __forceinline__ double &g(uint32_t k) const { return G[uint64_t(k) * 64 + lane]; }

    // adjoint of node j += c (or -= c) where `apply`; the first contribution
    // writes the whole row (0 + c, or 0 where the rule does not apply)
    __device__ __forceinline__ void contribute(uint32_t j, bool apply, double c, bool neg) const {
        const uint32_t f = flags(j);
        if (f & 1u) return;   // constants and observations take no adjoint
        double base = 0.0;
        if (f & 2u) {
            base = g(j);
        } else {
            set_flag(j, 2u);
        }
        const double nv = neg ? base - c : base + c;
        g(j) = apply ? nv : base;
    }
};

// Walk one work item (64 lanes of one program); returns false when a bound
// the host validation guarantees was not met (the lanes then hold NaN).
__device__ bool walk_item(const Args &A, const Wave &W, const ProgDesc &D, uint32_t q, int64_t l0) {
    const uint32_t lane = W.lane;
    const int64_t lg = l0 + lane;
    const bool active = lg < A.L;
    const int64_t lc = active ? lg : A.L - 1;
    const uint32_t *code = A.buf + D.code_off;
    const int32_t *match = reinterpret_cast<const int32_t *>(A.buf + D.match_off);
    const double *K = reinterpret_cast<const double *>(A.buf + D.const_off);
    const double *prm = A.params + int64_t(q) * A.prog_stride_p + lc * A.ld_p;
    const uint32_t n_nodes = D.n_nodes, P = D.n_params;
    if (n_nodes > A.n_nodes_max || D.depth > A.depth || D.n_locals > A.n_locals || D.n_loops > A.n_loops ||
        D.n_frames > A.n_frames)
        return false;

    for (uint32_t i = lane; i < (n_nodes + 15) / 16; i += 64) W.flg[i] = 0;
    for (uint32_t i = lane; i < D.n_locals; i += 64) W.loc[i] = kUnset;
    for (uint32_t p = 0; p < P; ++p) W.v(p) = prm[p];

    uint64_t mask = uni64(__ballot(active));
    uint32_t n = P, sp = 0, lp = 0, fp = 0, pc = 0, steps = 0;
    auto node = [&](uint32_t op, uint32_t a, uint32_t b) {
        Node e{op, a, b, 0, 0};
        W.E[n] = e;   // every lane stores the same record (each later reads its own store)
        return n++;
    };

    for (;;) {
        if (pc >= D.n_instr || ++steps > D.n_steps) return false;   // the walk always ends within both
        const uint32_t w0 = code[2 * pc], imm = code[2 * pc + 1];
        const uint32_t op = w0 & 0xFFu, wa = (w0 >> 8) & 0xFFu;
        // bounds the host validation guarantees (kept so that a broken
        // guarantee can only give NaN lanes, never an access out of bounds)
        uint32_t pops = 0, pushes = 0;
        stack_effect(op, &pops, &pushes);
        if (sp < pops || sp - pops + pushes > W.depth || (op == bc::LOOP && lp >= A.n_loops) ||
            (op == bc::IFLT && fp >= A.n_frames) || ((op == bc::ELSE || op == bc::ENDIF) && fp == 0) ||
            (op == bc::ENDLOOP && lp == 0))
            return false;
        switch (op) {
        case bc::HALT:
            goto reverse;
        case bc::PUSH:
            if (n >= n_nodes) return false;
            W.v(n) = K[imm];
            W.set_flag(n, 1u);
            W.stk[sp++] = node(walk::kLeaf, 0, 0);
            break;
        case bc::OBS: {
            if (n >= n_nodes || wa > lp) return false;
            int64_t idx = imm;
            for (uint32_t d = 0; d < wa; ++d)
                idx += int64_t(int32_t(code[2 * (pc + 1 + d) + 1])) * int64_t(uni(W.lps[3 * (lp - 1 - d) + 2]));
            W.v(n) = A.obs[idx];
            W.set_flag(n, 1u);
            W.stk[sp++] = node(walk::kLeaf, 0, 0);
            pc += wa;
            break;
        }
        case bc::PARAM:
            W.stk[sp++] = imm;
            break;
        case bc::LOADL: {
            const uint32_t id = uni(W.loc[imm]);
            if (id == kUnset) return false;
            W.stk[sp++] = id;
            break;
        }
        case bc::STOREL:
            W.loc[imm] = uni(W.stk[--sp]);
            break;
        case bc::DUP:
            W.stk[sp] = uni(W.stk[sp - 1]);
            ++sp;
            break;
        case bc::OVER:
            W.stk[sp] = uni(W.stk[sp - 2]);
            ++sp;
            break;
        case bc::SWAP: {
            const uint32_t t = uni(W.stk[sp - 1]), u = uni(W.stk[sp - 2]);
            W.stk[sp - 1] = u;
            W.stk[sp - 2] = t;
            break;
        }
        case bc::DROP:
            --sp;
            break;
        case bc::LOOP:
            if (imm == 0) {
                pc = uni(uint32_t(match[pc])) + 1;
                continue;
            }
            W.lps[3 * lp] = pc + 1;
            W.lps[3 * lp + 1] = imm;
            W.lps[3 * lp + 2] = 0;
            ++lp;
            break;
        case bc::ENDLOOP: {
            const uint32_t k = uni(W.lps[3 * (lp - 1) + 2]) + 1;
            if (k < uni(W.lps[3 * (lp - 1) + 1])) {
                W.lps[3 * (lp - 1) + 2] = k;
                pc = uni(W.lps[3 * (lp - 1)]);
                continue;
            }
            --lp;
            break;
        }
        case bc::IFLT: {
            const uint32_t bi = uni(W.stk[sp - 1]), ai = uni(W.stk[sp - 2]);
            sp -= 2;
            const uint64_t tm = uni64(__ballot(W.v(ai) < W.v(bi))) & mask, em = mask & ~tm;
            // frame: outer mask, first-arm mask, second-arm mask, phase, entry
            // depth, then the entry snapshot and the first arm's exit snapshot
            uint32_t *f = W.frm + fp * W.fsz;
            ++fp;
            f[0] = uint32_t(mask);
            f[1] = uint32_t(mask >> 32);
            f[2] = uint32_t(tm);
            f[3] = uint32_t(tm >> 32);
            f[4] = uint32_t(em);
            f[5] = uint32_t(em >> 32);
            f[6] = 0;
            f[7] = sp;
            for (uint32_t i = lane; i < sp; i += 64) f[walk::kFrameFixed + i] = W.stk[i];
            for (uint32_t i = lane; i < D.n_locals; i += 64) f[walk::kFrameFixed + W.depth + i] = W.loc[i];
            if (tm) {
                mask = tm;
                break;
            }
            mask = em;   // no lane takes the first arm: it is not walked
            pc = uni(uint32_t(match[pc])) + 1;
            continue;
        }
        case bc::ELSE: {   // end of a walked first arm
            uint32_t *f = W.frm + (fp - 1) * W.fsz;
            const uint64_t em = uint64_t(uni(f[4])) | uint64_t(uni(f[5])) << 32;
            f[6] = 1u | sp << 1;
            for (uint32_t i = lane; i < sp; i += 64) f[walk::kFrameFixed + W.snap + i] = W.stk[i];
            for (uint32_t i = lane; i < D.n_locals; i += 64) f[walk::kFrameFixed + W.snap + W.depth + i] = W.loc[i];
            if (em) {   // the second arm starts from the entry state
                sp = uni(f[7]);
                for (uint32_t i = lane; i < sp; i += 64) W.stk[i] = f[walk::kFrameFixed + i];
                for (uint32_t i = lane; i < D.n_locals; i += 64) W.loc[i] = f[walk::kFrameFixed + W.depth + i];
                mask = em;
                break;
            }
            pc = uni(uint32_t(match[pc]));   // to the ENDIF
            continue;
        }
        case bc::ENDIF: {
            const uint32_t *f = W.frm + (fp - 1) * W.fsz;
            const uint32_t ph = uni(f[6]);
            const uint64_t tm = uint64_t(uni(f[2])) | uint64_t(uni(f[3])) << 32;
            const uint64_t em = uint64_t(uni(f[4])) | uint64_t(uni(f[5])) << 32;
            if ((ph & 1u) && em) {   // both arms walked: merge what they left different
                if ((ph >> 1) != sp) return false;
                const bool first = (tm >> lane) & 1u;
                for (uint32_t i = 0; i < sp; ++i) {
                    const uint32_t x = uni(f[walk::kFrameFixed + W.snap + i]), y = uni(W.stk[i]);
                    if (x == y) continue;
                    if (n >= n_nodes) return false;
                    W.v(n) = first ? W.v(x) : W.v(y);
                    W.E[n] = Node{walk::kMerge, x, y, 0, tm};
                    W.stk[i] = n++;
                }
                for (uint32_t j = 0; j < D.n_locals; ++j) {
                    const uint32_t x = uni(f[walk::kFrameFixed + W.snap + W.depth + j]), y = uni(W.loc[j]);
                    if (x == y) continue;
                    if (x == kUnset || y == kUnset || n >= n_nodes) return false;
                    W.v(n) = first ? W.v(x) : W.v(y);
                    W.E[n] = Node{walk::kMerge, x, y, 0, tm};
                    W.loc[j] = n++;
                }
            }
            mask = uint64_t(uni(f[0])) | uint64_t(uni(f[1])) << 32;
            --fp;
            break;
        }
        default: {   // a scalar numeric word
            if (n >= n_nodes) return false;
            const bool bin = is_binary(op);
            const uint32_t bi = bin ? uni(W.stk[sp - 1]) : 0u;
            const uint32_t ai = uni(W.stk[sp - (bin ? 2 : 1)]);
            sp -= bin ? 2 : 1;
            W.v(n) = forward(op, W.v(ai), bin ? W.v(bi) : 0.0);
            W.stk[sp++] = node(op, ai, bi);
        }
        }
        ++pc;
    }

reverse: {
    const uint32_t loss_id = uni(W.stk[0]);
    const double loss = W.v(loss_id);
    W.contribute(loss_id, true, 1.0, false);   // seed: 0 + 1
    for (uint32_t k = n; k-- > P;) {
        if (W.flags(k) != 2u) continue;   // a leaf, or no adjoint reached it
        const Node e = W.E[k];
        const uint32_t op = uni(e.op), a = uni(e.a), b = uni(e.b);
        const double g = W.g(k);
        const bool on = g != 0.0;
        switch (op) {
        case walk::kMerge: {
            const bool first = (uni64(e.mask) >> lane) & 1u;
            W.contribute(a, on && first, g, false);
            W.contribute(b, on && !first, g, false);
            break;
        }
        case bc::ADD:
            W.contribute(a, on, g, false);
            W.contribute(b, on, g, false);
            break;
        case bc::SUB:
            W.contribute(a, on, g, false);
            W.contribute(b, on, g, true);
            break;
        case bc::MUL: {
            const double x = W.v(a), y = W.v(b);
            W.contribute(a, on, g * y, false);
            W.contribute(b, on, g * x, false);
            break;
        }
        case bc::DIV: {
            const double y = W.v(b), z = W.v(k);
            W.contribute(a, on, g / y, false);
            W.contribute(b, on, (g * z) / y, true);
            break;
        }
        case bc::NEG:
            W.contribute(a, on, g, true);
            break;
        case bc::EXP:
            W.contribute(a, on, g * W.v(k), false);
            break;
        case bc::LOG: {
            const double x = W.v(a);
            W.contribute(a, on && x > 1e-8, g / x, false);
            break;
        }
        case bc::SQRT: {
            const double x = W.v(a);
            W.contribute(a, on && x > 1e-8, g / (2.0 * W.v(k)), false);
            break;
        }
        case bc::SIN:
            W.contribute(a, on, g * cos(W.v(a)), false);
            break;
        case bc::COS:
            W.contribute(a, on, g * sin(W.v(a)), true);
            break;
        case bc::ABS: {
            const double x = W.v(a);
            W.contribute(a, on, x > 0.0 ? g : (x < 0.0 ? -g : 0.0), false);
            break;
        }
        default: {   // POW
            const double x = W.v(a), y = W.v(b), z = W.v(k);
            W.contribute(a, on, ((g * y) * z) / x, false);
            W.contribute(b, on, (g * z) * log(x), false);
        }
        }
    }
    if (active) {
        A.loss[int64_t(q) * A.L + lg] = loss;
        double *gr = A.grad + int64_t(q) * A.prog_stride_g + lg * A.ld_g;
        for (uint32_t p = 0; p < P; ++p) gr[p] = (W.flags(p) & 2u) ? W.g(p) : 0.0;
    }
}
    return true;
}

__global__ void __launch_bounds__(64) ndvm_walk(Args A) {
    extern __shared__ uint32_t sh[];
    Wave W;
    W.lane = threadIdx.x;
    W.depth = A.depth;
    W.snap = A.depth + A.n_locals;
    W.fsz = walk::kFrameFixed + 2 * W.snap;
    W.stk = sh;
    W.loc = W.stk + A.depth;
    W.lps = W.loc + A.n_locals;
    W.frm = W.lps + 3 * A.n_loops;
    W.flg = W.frm + A.n_frames * W.fsz;
    uint8_t *slot = A.ws + uint64_t(blockIdx.x) * A.n_nodes_max * walk::ws_bytes_per_node();
    W.V = reinterpret_cast<double *>(slot);
    W.G = W.V + uint64_t(A.n_nodes_max) * 64;
    W.E = reinterpret_cast<Node *>(W.G + uint64_t(A.n_nodes_max) * 64);
    const uint64_t per_prog = uint64_t((A.L + 63) / 64);
    const ProgDesc *descs = reinterpret_cast<const ProgDesc *>(A.buf);
    for (uint64_t item = blockIdx.x; item < A.n_items; item += gridDim.x) {
        const uint32_t q = uint32_t(item / per_prog);
        const int64_t l0 = int64_t(item % per_prog) * 64;
        const ProgDesc D = descs[q];
        if (!walk_item(A, W, D, q, l0)) {
            // a bound the validation guarantees was not met: report it and
            // leave this item's lanes NaN
            if (W.lane == 0) atomicOr(A.status, 1);
            const int64_t lg = l0 + W.lane;
            if (lg < A.L) {
                A.loss[int64_t(q) * A.L + lg] = NAN;
                double *gr = A.grad + int64_t(q) * A.prog_stride_g + lg * A.ld_g;
                for (uint32_t p = 0; p < D.n_params; ++p) gr[p] = NAN;
            }
        }
    }
}

}  // namespace

hipError_t launch_walk(const walk::Args &A, uint32_t grid, hipStream_t stream) {
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(ndvm_walk, dim3(grid), dim3(64), size_t(A.lds_words) * 4, stream, A);
    return hipGetLastError();
}

}  // namespace ndvm
