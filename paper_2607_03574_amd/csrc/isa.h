// Device program format executed by the replay kernel.  Produced by the
// scheduler from a validated tape; not part of the public interface.
//
// A program is a sequence of 8-word instructions.  Each lane owns a file of
// fp64 "registers" (lane values and adjoints); register r of lane l lives in
// LDS when r < R_lds and in the workspace spill area otherwise.
//
//   w0 : op (bits 0-7) | mode (8-15) | nel (16-23)
//   w1 : destination register (forward) / adjoint register g of the output
//        (reverse)
//   w2, w3 : operands a, b     w4 : operand c / output value z (reverse)
//   w5 : operand d (select) / adjoint target of a (reverse)
//   w6 : adjoint target of b (reverse)
//   w7 : immediate (dims, element index, aux offset, checkpoint row, param)
//
// Operand words are register indices: constants (the tape's pool and the
// constants 1, -1, -0 that bundles use) are loaded into static registers once
// (LDCONST) and observations by LDOBS where they are used.
// Adjoint target words: register | kInit (first contribution: store instead
// of add), or kNone (generic handlers; scalar handlers get a sink register).
#pragma once
#include <cstdint>

namespace ndvm {
namespace isa {

enum : uint32_t {
    END = 0,
    LDPARAM = 1,   // w1 dst, w7 param index
    ST_LOSS = 2,   // w2 operand
    CKPT_ST = 3,   // w2 src reg, w7 checkpoint row, nel
    CKPT_LD = 4,   // w1 dst reg, w7 checkpoint row, nel
    ZERO = 5,      // w1 dst reg, nel
    SEED = 6,      // w5 target
    ST_GRAD = 7,   // w2 src reg, w7 param index
    LDOBS = 8,     // w1 dst, w7 observation index
    LDCONST = 9,   // w1 dst, w7 first pool entry, nel entries
    NOP = 10,      // padding before the END that opens the program's last chunk
    // N = 2..4 observation loads: word k + 1 = destination | index << 16
    OB2 = 11, OB3 = 12, OB4 = 13,

    F_ADD = 16, F_SUB, F_MUL, F_DIV, F_NEG, F_EXP, F_LOG, F_SQRT, F_SIN, F_COS, F_ABS, F_POW,
    F_DOT, F_MATMUL, F_TRANSPOSE, F_TRACE, F_INV, F_DET, F_LOGDET, F_OUTER, F_PACK, F_INDEX,
    F_SELECT,

    R_ADD = 48, R_SUB, R_MUL, R_DIV, R_NEG, R_EXP, R_LOG, R_SQRT, R_SIN, R_COS, R_ABS, R_POW,
    R_DOT, R_MATMUL, R_TRANSPOSE, R_TRACE, R_INV, R_DET, R_LOGDET, R_OUTER, R_PACK, R_INDEX,
    R_SELECT,

    // scalar (1x1) fast paths of the elementwise ops and the select: no
    // element loops, no broadcast modes
    S_ADD = 96, S_SUB, S_MUL, S_DIV, S_NEG, S_EXP, S_LOG, S_SQRT, S_SIN, S_COS, S_ABS, S_SELECT,
    SR_ADD = 112, SR_SUB, SR_MUL, SR_DIV, SR_NEG, SR_EXP, SR_LOG, SR_SQRT, SR_SIN, SR_COS, SR_ABS,
    SR_SELECT,

    // Bundles: N = 1..3 independent scalar ops or adjoint rules in one
    // instruction, each a run of 16-bit register fields (field i < 14 is half
    // i & 1 of word 1 + i / 2, field 14 the high half of w0).  First
    // contributions of adjoint rules are flagged in w0: bit 8 + 2k for rule
    // k's target a, bit 9 + 2k for its target b.
    // Sums, differences, products and negations all become one fused
    // multiply-add against the constant registers 1, -1 and -0, which gives
    // the same bits as the plain operation:
    //   a + b = fma(a, 1, b)   a - b = fma(b, -1, a)   a * b = fma(a, b, -0)
    //   -a = fma(a, -1, -0)
    FB1 = 128, FB2, FB3,      // fields (d, x, y, w) per op: d = fma(x, y, w)
    DB1, DB2, DB3,            // fields (d, a, b) per op: d = a / b
    // linear adjoint rules, fields (g, ya, yb, ta, tb): ta += g * ya,
    // tb += g * yb, gated on g != 0 (add: 1, 1; sub: 1, -1; mul: b, a;
    // neg: -1 with tb the sink; exp: z with tb the sink)
    LB1, LB2, LB3,
    // division adjoint rules, fields (g, b, z, ta, tb): ta += g / b,
    // tb += -((g * z) / b), gated on g != 0
    RDB1, RDB2, RDB3,
    // the same with targets that may repeat (x * x, or two rules feeding one
    // adjoint): each target is read after the previous rule has written it
    LBS1, LBS2, LBS3, RDBS1, RDBS2, RDBS3,
    OP_COUNT
};

// binary elementwise broadcast modes (w0 bits 8-15)
enum : uint32_t { MODE_SAME = 0, MODE_A_SCALAR = 1, MODE_B_SCALAR = 2 };

constexpr uint32_t kIndexMask = (1u << 30) - 1;
constexpr uint32_t kInit = 0x80000000u;
constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr uint32_t kWords = 8;
// The program is fetched in chunks of 32 instructions (one 16-byte load per
// thread of a wave).  Its END is the first instruction of a chunk (NOPs pad
// the chunk before), and one more chunk of END follows, which the fetch reads
// ahead; so the replay loop tests for END once per chunk.
constexpr uint32_t kChunkInstr = 32;
constexpr uint32_t kChunkWords = kChunkInstr * kWords;
constexpr uint32_t kFieldMaxReg = 1u << 16;   // registers addressable by bundle fields
// Set on a bundle, observation bundle or matmul when the next instruction has
// the same opcode and lies in the same fetch chunk: the handler runs it too,
// without going back through the dispatch.
constexpr uint32_t kRepeat = 1u << 15;

inline uint32_t w0(uint32_t op, uint32_t mode, uint32_t nel) { return op | (mode << 8) | (nel << 16); }
inline uint32_t dims(uint32_t m, uint32_t k, uint32_t n) { return m | (k << 8) | (n << 16); }

}  // namespace isa

// Per-program constants read by the kernel: the device program and where the
// program's checkpoint and spill rows start in the workspace.  Depends only
// on the program and the launch's register budget, never on per-call
// pointers, so a table of these can be cached on the device.
struct ProgStatic {
    const uint32_t *prog;    // instruction words
    const uint32_t *aux;     // operand / target lists
    const double *consts;    // constant pool
    uint64_t ckpt_row0;      // checkpoint row r of lane l at ws[(ckpt_row0 + r)*Lpad + l]
    uint64_t spill_row0;     // register r_lds + r of lane l at ws[(spill_row0 + r)*Lpad + l]
    uint32_t r_lds;          // registers held in LDS
    uint32_t spills;         // nonzero when the program has registers beyond r_lds
};

// Kernel variant of a launch: every register in LDS, a spill tail for every
// program, or chosen per program (many-program launches that mix the two).
enum LaunchVariant : int { kLdsOnly = 0, kSpill = 1, kPerProgram = 2 };

// Per-call arguments.  Program q of a launch (blockIdx.y) reads
// params + q*prog_stride_p and writes loss + q*L, grad + q*prog_stride_g.
struct LaunchArgs {
    const double *obs;
    const double *params;
    double *loss;
    double *grad;
    double *ws;
    int64_t ld_p, ld_g, L, Lpad, prog_stride_p, prog_stride_g;
};

}  // namespace ndvm
