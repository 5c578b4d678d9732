// Device walker kernel: the structural walk of a stack-bytecode program on
// the GPU, one wave per 64 lanes of one program (definitions and layout in
// walk.h).
//
// Control is the same for every lane of a wave: program counter, operand
// stack (node numbers), locals, loop counters and branch frames live once
// per wave in LDS and are read back as wave-uniform values.  Numbers are
// per lane.  The forward walk keeps the operand stack's and the locals'
// values in LDS rows (one double per lane), so a word reads its operands
// there; every node it records is also stored, as a coalesced row of 64
// doubles, to the wave's slot in HBM for the reverse sweep.  A numeric IFLT
// takes one ballot: each arm runs under the mask of the lanes that take it,
// an arm no lane takes is not walked at all, and when both arms ran their
// differing stack positions and locals become MERGE nodes (Section 6, lane
// masking).  The reverse sweep visits the recorded nodes from last to first
// and applies the adjoint rules of Appendix C, table tab:adjoints, per lane,
// gated on a nonzero incoming adjoint; an adjoint row is written in full by
// its first contribution (zero where the rule does not apply), so no row is
// cleared beforehand, and a node no rule reached is skipped without a read.
// The parameters' values and adjoints stay in LDS.
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

// Read-only inputs (the program buffer, the observations) are read through
// the constant address space, so wave-uniform reads become scalar loads that
// wait for nothing else (a vector load would wait for every store the walk
// has in flight before it).
#define AS_CONST __attribute__((address_space(4)))
template <class T>
__device__ __forceinline__ const AS_CONST T *cst(const T *p) {
    return (const AS_CONST T *)(p);
}

__device__ __forceinline__ uint32_t uni(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint64_t uni64(uint64_t v) {
    return uint64_t(uni(uint32_t(v))) | uint64_t(uni(uint32_t(v >> 32))) << 32;
}

__device__ __forceinline__ double clampv(double x) { return x < 1e-8 ? 1e-8 : x; }

__device__ __forceinline__ bool is_binary(uint32_t op) {
    return op == bc::ADD || op == bc::SUB || op == bc::MUL || op == bc::DIV || op == bc::POW;
}

// Library transcendentals, one call site each (inlined: an out-of-line call
// would wait for every store the walk has in flight at its entry; measured
// 4% slower on the random-program population despite the registers saved).
__device__ __forceinline__ double transcendental(uint32_t op, double x, double y) {
    switch (op) {
    case bc::EXP: return exp(x);
    case bc::LOG: return log(x);
    case bc::SIN: return sin(x);
    case bc::COS: return cos(x);
    default: return pow(x, y);
    }
}

// forward value of a scalar word
__device__ __forceinline__ double forward(uint32_t op, double x, double y) {
    switch (op) {
    case bc::ADD: return x + y;
    case bc::SUB: return x - y;
    case bc::MUL: return x * y;
    case bc::DIV: return x / y;
    case bc::NEG: return -x;
    case bc::SQRT: return sqrt(clampv(x));
    case bc::ABS: return fabs(x);
    case bc::LOG: return transcendental(bc::LOG, clampv(x), 0.0);
    default: return transcendental(op, x, y);   // EXP SIN COS POW
    }
}

struct Wave {
    uint32_t lane;
    uint32_t P;   // parameters of the current program
    // LDS: value rows (64 doubles each)
    double *VP;   // parameters' values
    double *VS;   // operand stack values (forward)
    double *VL;   // locals' values (forward)
    double *GP;   // parameters' adjoints (reverse; the rows of VS and VL)
    // LDS: structural words
    uint32_t *stk, *loc, *lps, *frm, *flg;
    uint32_t snap, fsz, depth;
    // HBM slot of the wave
    double *V, *G;
    Node *E;
    uint64_t *M;   // ballot words of MERGE nodes

    // one flag bit per node in LDS: its adjoint row has been written
    __device__ __forceinline__ bool touched(uint32_t k) const { return (uni(flg[k >> 5]) >> (k & 31)) & 1u; }
    __device__ __forceinline__ void touch(uint32_t k) const {
        const uint32_t w = uni(flg[k >> 5]);
        flg[k >> 5] = w | 1u << (k & 31);
    }
    __device__ __forceinline__ double &s(uint32_t i) const { return VS[i * 64 + lane]; }
    __device__ __forceinline__ double &l(uint32_t j) const { return VL[j * 64 + lane]; }
    // value and adjoint of node k (parameters in LDS, the others in HBM;
    // a leaf's number carries kLeafBit)
    __device__ __forceinline__ double &v(uint32_t k) const {
        k &= ~walk::kLeafBit;
        return k < P ? VP[k * 64 + lane] : V[k * 64u + lane];
    }
    __device__ __forceinline__ double &g(uint32_t k) const {
        return k < P ? GP[k * 64 + lane] : G[k * 64u + lane];
    }

    // adjoint of node j += c (or -= c) where `apply`; the first contribution
    // writes the whole row (0 + c, or 0 where the rule does not apply)
    __device__ __forceinline__ void contribute(uint32_t j, bool apply, double c, bool neg) const {
        if (j & walk::kLeafBit) return;   // constants and observations take no adjoint
        double base = 0.0;
        if (touched(j)) {
            base = g(j);
        } else {
            touch(j);
        }
        const double nv = neg ? base - c : base + c;
        g(j) = apply ? nv : base;
    }
};

// Walk one work item (64 lanes of one program); returns false when a bound
// the host validation guarantees was not met (the lanes then hold NaN).
__device__ bool walk_item(const Args &A, Wave &W, const ProgDesc &D, uint32_t q, int64_t l0) {
    const uint32_t lane = W.lane;
    const int64_t lg = l0 + lane;
    const bool active = lg < A.L;
    const int64_t lc = active ? lg : A.L - 1;
    const AS_CONST uint32_t *code = cst(A.buf + D.code_off);
    const AS_CONST int32_t *match = cst(reinterpret_cast<const int32_t *>(A.buf + D.match_off));
    const AS_CONST double *K = cst(reinterpret_cast<const double *>(A.buf + D.const_off));
    const AS_CONST double *obs = cst(A.obs);
    const double *prm = A.params + int64_t(q) * A.prog_stride_p + lc * A.ld_p;
    const uint32_t n_nodes = D.n_nodes, P = D.n_params;
    if (n_nodes > A.n_nodes_max || D.depth > A.depth || D.n_locals > A.n_locals || D.n_loops > A.n_loops ||
        D.n_frames > A.n_frames || P > A.n_params)
        return false;
    W.P = P;

    for (uint32_t i = lane; i < (n_nodes + 31) / 32; i += 64) W.flg[i] = 0;
    for (uint32_t i = lane; i < D.n_locals; i += 64) W.loc[i] = kUnset;
    for (uint32_t p = 0; p < P; ++p) W.VP[p * 64 + lane] = prm[p];

    uint64_t mask = uni64(__ballot(active));
    uint32_t n = P, sp = 0, lp = 0, fp = 0, pc = 0, steps = 0;
    // record node n (every lane stores the same record: each later reads its own store)
    auto record = [&](uint32_t op, uint32_t a, uint32_t b, double val) {
        W.V[n * 64u + lane] = val;
        W.E[n] = Node{op, a, b, 0};
        return n++;
    };
    // restore the stack and locals values of an IFLT's entry state (node
    // numbers in the frame snapshot) wherever the current state differs
    auto restore = [&](const uint32_t *snap_ids, uint32_t sp0, uint32_t sp_now) {
        for (uint32_t i = 0; i < sp0; ++i) {
            const uint32_t x = uni(snap_ids[i]);
            if (i < sp_now && uni(W.stk[i]) == x) continue;
            W.stk[i] = x;
            W.s(i) = W.v(x);
        }
        for (uint32_t j = 0; j < D.n_locals; ++j) {
            const uint32_t x = uni(snap_ids[W.depth + j]);
            if (uni(W.loc[j]) == x) continue;
            W.loc[j] = x;
            if (x != kUnset) W.l(j) = W.v(x);
        }
    };

    for (;;) {
        if (pc >= D.n_instr || ++steps > D.n_steps) return false;   // the walk always ends within both
        const uint32_t w0 = code[2 * pc], imm = code[2 * pc + 1];
        const uint32_t op = w0 & 0xFFu, wa = (w0 >> 8) & 0xFFu;
        // bounds the host validation guarantees (kept so that a broken
        // guarantee can only give NaN lanes, never an access out of bounds);
        // the host packs each word's stack effect into it
        const uint32_t pops = (w0 >> 16) & 3u, pushes = (w0 >> 18) & 3u;
        if (sp < pops || sp - pops + pushes > W.depth) return false;   // the other bounds: in their words
        switch (op) {
        case bc::HALT:
            goto reverse;
        case bc::PUSH: {
            if (n >= n_nodes) return false;
            const double x = K[imm];
            W.s(sp) = x;
            W.stk[sp++] = record(walk::kLeaf, 0, 0, x) | walk::kLeafBit;
            break;
        }
        case bc::OBS: {
            if (n >= n_nodes || wa > lp) return false;
            int64_t idx = imm;
            for (uint32_t d = 0; d < wa; ++d)
                idx += int64_t(int32_t(code[2 * (pc + 1 + d) + 1])) * int64_t(uni(W.lps[3 * (lp - 1 - d) + 2]));
            const double x = obs[idx];
            W.s(sp) = x;
            W.stk[sp++] = record(walk::kLeaf, 0, 0, x) | walk::kLeafBit;
            pc += wa;
            break;
        }
        case bc::PARAM:
            if (imm >= P) return false;
            W.s(sp) = W.VP[imm * 64 + lane];
            W.stk[sp++] = imm;
            break;
        case bc::LOADL: {
            if (imm >= D.n_locals) return false;
            const uint32_t id = uni(W.loc[imm]);
            if (id == kUnset) return false;
            W.s(sp) = W.l(imm);
            W.stk[sp++] = id;
            break;
        }
        case bc::STOREL:
            if (imm >= D.n_locals) return false;
            --sp;
            W.l(imm) = W.s(sp);
            W.loc[imm] = uni(W.stk[sp]);
            break;
        case bc::DUP:
            W.s(sp) = W.s(sp - 1);
            W.stk[sp] = uni(W.stk[sp - 1]);
            ++sp;
            break;
        case bc::OVER:
            W.s(sp) = W.s(sp - 2);
            W.stk[sp] = uni(W.stk[sp - 2]);
            ++sp;
            break;
        case bc::SWAP: {
            const double x = W.s(sp - 1), y = W.s(sp - 2);
            const uint32_t t = uni(W.stk[sp - 1]), u = uni(W.stk[sp - 2]);
            W.s(sp - 1) = y;
            W.s(sp - 2) = x;
            W.stk[sp - 1] = u;
            W.stk[sp - 2] = t;
            break;
        }
        case bc::DROP:
            --sp;
            break;
        case bc::LOOP:
            if (lp >= A.n_loops) return false;
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
            if (lp == 0) return false;
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
            if (fp >= A.n_frames) return false;
            sp -= 2;
            const uint64_t tm = uni64(__ballot(W.s(sp) < W.s(sp + 1))) & mask, em = mask & ~tm;
            // frame: outer mask, first-arm mask, second-arm mask, phase, entry
            // depth, then the entry snapshot and the first arm's exit snapshot
            // (node numbers of stack positions and locals)
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
            if (fp == 0) return false;
            uint32_t *f = W.frm + (fp - 1) * W.fsz;
            const uint64_t em = uint64_t(uni(f[4])) | uint64_t(uni(f[5])) << 32;
            f[6] = 1u | sp << 1;
            for (uint32_t i = lane; i < sp; i += 64) f[walk::kFrameFixed + W.snap + i] = W.stk[i];
            for (uint32_t i = lane; i < D.n_locals; i += 64) f[walk::kFrameFixed + W.snap + W.depth + i] = W.loc[i];
            if (em) {   // the second arm starts from the entry state
                const uint32_t sp0 = uni(f[7]);
                restore(f + walk::kFrameFixed, sp0, sp);
                sp = sp0;
                mask = em;
                break;
            }
            pc = uni(uint32_t(match[pc]));   // to the ENDIF
            continue;
        }
        case bc::ENDIF: {
            if (fp == 0) return false;
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
                    const double val = first ? W.v(x) : W.s(i);
                    W.V[n * 64u + lane] = val;
                    W.E[n] = Node{walk::kMerge, x, y, 0};
                    W.M[n] = tm;
                    W.s(i) = val;
                    W.stk[i] = n++;
                }
                for (uint32_t j = 0; j < D.n_locals; ++j) {
                    const uint32_t x = uni(f[walk::kFrameFixed + W.snap + W.depth + j]), y = uni(W.loc[j]);
                    if (x == y) continue;
                    if (x == kUnset || y == kUnset || n >= n_nodes) return false;
                    const double val = first ? W.v(x) : W.l(j);
                    W.V[n * 64u + lane] = val;
                    W.E[n] = Node{walk::kMerge, x, y, 0};
                    W.M[n] = tm;
                    W.l(j) = val;
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
            const double x = W.s(sp - (bin ? 2 : 1)), y = bin ? W.s(sp - 1) : 0.0;
            sp -= bin ? 2 : 1;
            const double z = forward(op, x, y);
            W.s(sp) = z;
            W.stk[sp++] = record(op, ai, bi, z);
        }
        }
        ++pc;
    }

reverse: {
    const uint32_t loss_id = uni(W.stk[0]);
    const double loss = W.s(0);
    W.contribute(loss_id, true, 1.0, false);   // seed: 0 + 1
    // the next node's record is loaded one node ahead
    Node nx = n > P ? W.E[n - 1] : Node{};
    for (uint32_t k = n; k-- > P;) {
        const Node e = nx;
        if (k > P) nx = W.E[k - 1];
        if (!W.touched(k)) continue;   // a leaf, or no adjoint reached it
        const uint32_t op = uni(e.op), a = uni(e.a), b = uni(e.b);
        // Every load the node's rules need is issued before the first
        // contribution is formed (the incoming adjoint, the values the rule
        // reads, the targets' adjoint rows), so the node waits on memory
        // once; a target named twice (x * x) takes its second contribution
        // on top of the first.
        const bool two = is_binary(op) || op == walk::kMerge;
        const bool need_x = op == bc::MUL || op == bc::LOG || op == bc::SQRT || op == bc::SIN || op == bc::COS ||
                            op == bc::ABS || op == bc::POW;
        const bool need_y = op == bc::MUL || op == bc::DIV || op == bc::POW;
        const bool need_z = op == bc::DIV || op == bc::EXP || op == bc::SQRT || op == bc::POW;
        const double g = W.g(k);
        const double x = need_x ? W.v(a) : 0.0, y = need_y ? W.v(b) : 0.0, z = need_z ? W.v(k) : 0.0;
        const bool has_a = !(a & walk::kLeafBit), has_b = two && !(b & walk::kLeafBit);
        const bool ta = has_a && W.touched(a), tb = has_b && b != a && W.touched(b);
        const double ga = ta ? W.g(a) : 0.0, gb = tb ? W.g(b) : 0.0;
        const bool on = g != 0.0;
        // contributions: value, where it applies, subtracted
        double ca = 0.0, cb = 0.0;
        bool pa = on, pb = on, na = false, nb = false;
        switch (op) {
        case walk::kMerge: {
            const bool first = (uni64(W.M[k]) >> lane) & 1u;
            ca = cb = g;
            pa = on && first;
            pb = on && !first;
            break;
        }
        case bc::ADD:
            ca = cb = g;
            break;
        case bc::SUB:
            ca = cb = g;
            nb = true;
            break;
        case bc::MUL:
            ca = g * y;
            cb = g * x;
            break;
        case bc::DIV:
            ca = g / y;
            cb = (g * z) / y;
            nb = true;
            break;
        case bc::NEG:
            ca = g;
            na = true;
            break;
        case bc::EXP:
            ca = g * z;
            break;
        case bc::LOG:
            pa = on && x > 1e-8;
            ca = g / x;
            break;
        case bc::SQRT:
            pa = on && x > 1e-8;
            ca = g / (2.0 * z);
            break;
        case bc::SIN:
            ca = g * transcendental(bc::COS, x, 0.0);
            break;
        case bc::COS:
            ca = g * transcendental(bc::SIN, x, 0.0);
            na = true;
            break;
        case bc::ABS:
            ca = x > 0.0 ? g : (x < 0.0 ? -g : 0.0);
            break;
        default:   // POW
            ca = ((g * y) * z) / x;
            cb = (g * z) * transcendental(bc::LOG, x, 0.0);
        }
        // the first contribution to a row writes it whole (0 + c, or 0
        // where the rule does not apply)
        double ra = 0.0;
        if (has_a) {
            if (!ta) W.touch(a);
            const double nv = na ? ga - ca : ga + ca;
            ra = pa ? nv : ga;
            W.g(a) = ra;
        }
        if (has_b) {
            const double base = b == a ? ra : gb;
            if (b != a && !tb) W.touch(b);
            const double nv = nb ? base - cb : base + cb;
            W.g(b) = pb ? nv : base;
        }
    }
    if (active) {
        A.loss[int64_t(q) * A.L + lg] = loss;
        double *gr = A.grad + int64_t(q) * A.prog_stride_g + lg * A.ld_g;
        for (uint32_t p = 0; p < P; ++p) gr[p] = W.touched(p) ? W.GP[p * 64 + lane] : 0.0;
    }
}
    return true;
}

__global__ void __launch_bounds__(64) ndvm_walk(Args A) {
    extern __shared__ double sh[];
    Wave W;
    W.lane = threadIdx.x;
    W.depth = A.depth;
    W.snap = A.depth + A.n_locals;
    W.fsz = walk::kFrameFixed + 2 * W.snap;
    W.VP = sh;
    W.VS = W.VP + A.n_params * 64;
    W.VL = W.VS + A.depth * 64;
    W.GP = W.VS;
    uint32_t *words = reinterpret_cast<uint32_t *>(sh + walk::lds_rows(A.depth, A.n_locals, A.n_params) * 64);
    W.stk = words;
    W.loc = W.stk + A.depth;
    W.lps = W.loc + A.n_locals;
    W.frm = W.lps + 3 * A.n_loops;
    W.flg = W.frm + A.n_frames * W.fsz;
    uint8_t *slot = A.ws + uint64_t(blockIdx.x) * A.n_nodes_max * walk::ws_bytes_per_node();
    W.V = reinterpret_cast<double *>(slot);
    W.G = W.V + uint64_t(A.n_nodes_max) * 64;
    W.E = reinterpret_cast<Node *>(W.G + uint64_t(A.n_nodes_max) * 64);
    W.M = reinterpret_cast<uint64_t *>(W.E + A.n_nodes_max);
    const uint64_t per_prog = uint64_t((A.L + 63) / 64);
    const AS_CONST uint32_t *descs = cst(A.buf);   // ProgDesc records, word by word
    for (uint64_t item = blockIdx.x; item < A.n_items; item += gridDim.x) {
        const uint32_t q = uint32_t(item / per_prog);
        const int64_t l0 = int64_t(item % per_prog) * 64;
        ProgDesc D;
        uint32_t *dw = reinterpret_cast<uint32_t *>(&D);
        for (uint32_t i = 0; i < sizeof(ProgDesc) / 4; ++i) dw[i] = descs[uint64_t(q) * (sizeof(ProgDesc) / 4) + i];
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
    hipLaunchKernelGGL(ndvm_walk, dim3(grid), dim3(64), size_t(A.lds_bytes), stream, A);
    return hipGetLastError();
}

}  // namespace ndvm
