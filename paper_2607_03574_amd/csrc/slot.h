// Device program format of the replay kernel ("slot" programs).  Produced by
// the scheduler from a validated tape; not part of the public interface.
//
// A wave of 64 threads replays 64/S lanes (parameter vectors) with S slots
// each: thread t serves lane t % (64/S) in slot t / (64/S).  Every
// instruction carries one micro-op per slot, all of the same form; the slots
// of one lane run independent micro-ops side by side, so a lane's
// instruction-level parallelism becomes thread parallelism and the wave count
// of a launch grows S-fold.
//
// Each lane owns a file of fp64 registers in LDS (register r of lane l at
// lds[r * (64/S) + l]); registers past the LDS budget live in lane-contiguous
// workspace rows.  A micro-op reads its operands from the file, computes one
// fp64 result and writes it back.  All slots of an instruction read before
// any slot writes, so the slots of one instruction never depend on each other.
//
// Per slot and instruction: four 32-bit words.
//   w0: bits 0-23 register a (destination, adjoint target or stored source)
//       bits 24-29 form (the same in every slot)
//       bit 30 kGated: the contribution is skipped when operand x is zero
//       bit 31 kFirst: first contribution to the target (store, do not add)
//   w1..w3: bits 0-23 operand fields x, y, z (registers or indices)
//       bits 24-31 uniform immediates i1, i2, i3 (the same in every slot)
// Slots an instruction does not use hold a copy of slot 0's micro-op whose
// result goes to the sink register (and whose checkpoint store goes to the
// trash row); forms with side effects outside the register file mask them.
#pragma once
#include <cstdint>

namespace ndvm {
namespace slot {

// Contribution rule of the adjoint forms: base = (kFirst ? +0 : t), then
// t = gate ? base + contribution : base, one rounding per operation.
enum Form : uint32_t {
    // ---- hot forms: no per-lane control flow
    // d = x * y + z (product rounded, then sum rounded).  Sums, differences,
    // products, negations and copies are this form against the constants
    // 1, -1, -0, with the bits of the plain operation.
    MAC = 1,
    ACC,       // t = (!kGated || x != 0) ? base + x * y : base, z = t: the linear adjoint rule t += g * y
    MACG,      // t = gate(z) ? base + x * y : base          (explicit gate register z)
    DIV,       // d = x / y
    ACCD,      // t = gate(z) ? base + x / y : base
    ACCND,     // t = gate(z) ? base + -(x / y) : base
    DOT,       // d = fma chain over k < i1 of A[x + k*i2] * B[y + k*i3], ascending, first term a product
    DOTACC,    // t = gate(z) ? base + (+/-)dot : base   (dot as DOT; i1 bit 7 negates)
    CMPLT,     // d = x < y ? 1 : 0   (unordered -> 0)
    SELP,      // d = p(x) != 0 ? y : z
    ACCSEL,    // t = gate(z) != 0 && (p(y) != 0) == i1 ? base + x : base
    DET2,      // d = A0 * A3 - A1 * A2 for the 2x2 matrix at x (two products, then difference)
    NZ,        // d = any of x .. x + i1 - 1 nonzero ? 1 : 0
    GATEGT,    // d = gate(z) != 0 && x > y ? 1 : 0
    ACCABS,    // t = gate(z) ? base + (y > 0 ? x : y < 0 ? -x : 0) : base
    SUMK,      // d = ((A[x] + A[x + i2]) + A[x + 2 i2]) ... over k < i1
    LDOBS,     // d = obs[x]
    LDPARAM,   // d = params[lane, x]
    LDCONST,   // d = consts[x]
    CKST,      // ckpt row x of this lane = register a
    CKLD,      // d = ckpt row x of this lane
    ZERO,      // d = +0
    HOT_END,
    // ---- cold forms: library transcendentals (per-lane branches) and
    // stores outside the register file
    UN = 40,   // d = f(x), f = i1: see Unary
    POW,       // d = pow(x, y)
    STLOSS,    // loss[lane] = register a          (slots < i1 only)
    STGRAD,    // grad[lane, x] = register a       (slots < i1 only)
    END = 63,
};

enum Unary : uint32_t { U_EXP = 0, U_LOGC, U_SQRTC, U_SIN, U_COS, U_ABS, U_LOG };

constexpr uint32_t kFieldMask = (1u << 24) - 1;
constexpr uint32_t kGated = 1u << 30;
constexpr uint32_t kFirst = 1u << 31;
constexpr uint32_t kFormShift = 24;
constexpr uint32_t kMaxField = kFieldMask;   // largest register / index a field holds
constexpr uint32_t kNegate = 0x80;           // DOTACC: subtract the dot product

// Program fetch: a chunk holds kChunk instructions as 4 rows x kChunk x 4
// words; row r (threads 16r .. 16r + 15 of a wave) carries the micro-ops of
// slot r * S / 4, and thread 16r + j holds word j of its row (instruction
// j / 4, word j % 4), so one coalesced dword load per thread fetches the
// chunk and a row broadcast hands every thread of a slot its words.  The
// program is padded so that the chunk holding END is followed by two more
// chunks (the fetch reads two ahead).  Slot counts 1, 2 and 4 (a slot's
// threads fill whole rows).
constexpr uint32_t kChunk = 4;
constexpr uint32_t kRows = 4;
constexpr uint32_t kChunkWords = kRows * kChunk * 4;
constexpr uint32_t kFetchAhead = 2;
constexpr uint32_t kMaxSlots = 4;

inline uint32_t form_of(uint32_t w0) { return (w0 >> kFormShift) & 63u; }
inline uint32_t word0(uint32_t form, uint32_t a, uint32_t flags = 0) { return a | (form << kFormShift) | flags; }
inline uint32_t fieldw(uint32_t f, uint32_t imm = 0) { return f | (imm << 24); }

inline bool is_hot(uint32_t form) { return form >= MAC && form < HOT_END; }
// forms whose register a is written
inline bool writes_a(uint32_t form) { return form != CKST && form != STLOSS && form != STGRAD && form != END; }

}  // namespace slot

// Per-program constants read by the kernel: the device program and where the
// program's checkpoint and spill rows start in the workspace.  Depends only
// on the program and the launch's register budget, never on per-call
// pointers, so a table of these can be cached on the device.
struct ProgStatic {
    const uint32_t *prog;    // payload words, chunk-major: [chunk][row][instr][4]
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
