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
// Per instruction: a header word, the same for every slot:
//   bits 0-5 form, bits 6-9 kFirst of slots 0-3 (first contribution to the
//   target: store, do not add), bit 10 set when the form is MAC, bit 11 when
//   it is ACC, bit 12 when it is MSUB, bit 13 when it is DOTB or DOTBACC (the
//   most frequent forms, each told apart by one bit test), bits 14-31 the
//   form's immediate;
// and per slot four words a, x, y, z: a register named in a field is held as
// its byte offset in a lane's register file (register * 8 * 64/S), an index
// (observation, parameter, constant, checkpoint row) as itself.
// Slots an instruction does not use hold a copy of slot 0's micro-op whose
// results go to the sink registers (and whose checkpoint stores go to the
// trash rows); forms with side effects outside the register file mask them.
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
    ACC,       // d = x != 0 ? z + x * y : z: the linear adjoint rule t += g * y gated on g, with
               // z = t, or z = a register holding +0 for the first contribution (d = t)
    MACG,      // t = gate(z) ? base + x * y : base          (explicit gate register z)
    DIV,       // d = x / y
    ACCD,      // t = gate(z) ? base + x / y : base
    ACCND,     // t = gate(z) ? base + -(x / y) : base
    DOT,       // d = fma chain over k < K of A[x + k sa] * B[y + k sb], ascending, first term a product
    DOTACC,    // t = gate(z) ? base + (+/-)dot : base   (dot as DOT)
    CMPLT,     // d = x < y ? 1 : 0   (unordered -> 0)
    SELP,      // d = p(x) != 0 ? y : z
    ACCSEL,    // t = gate(z) != 0 && (p(y) != 0) == imm ? base + x : base
    DET2,      // d = A0 * A3 - A1 * A2 for the 2x2 matrix at x (two products, then difference)
    NZ,        // d = any of x .. x + imm - 1 nonzero ? 1 : 0
    GATEGT,    // d = gate(z) != 0 && x > y ? 1 : 0
    ACCABS,    // t = gate(z) ? base + (y > 0 ? x : y < 0 ? -x : 0) : base
    SUMK,      // d = ((A[x] + A[x + s]) + A[x + 2 s]) ... over k < K  (imm = K | s << 6)
    ZERO,      // d = +0
    // block of N outputs d[c] = fma chain over k < K of X[x + k sx] * Y[y + k sy + c sc]
    // (ascending, first term a product)
    DOTB,
    DOTBACC,   // t[c] = gate(z) ? base[c] + (+/-)dot[c] : base[c]
    EXPF,      // d = exp(x)      (library functions without per-lane branches)
    LOGCF,     // d = log(max(x, 1e-8)) with x < 1e-8 -> 1e-8 (NaN propagates)
    LOGF,      // d = log(x)
    SQRTCF,    // d = sqrt(max(x, 1e-8)), clamped as LOGCF
    ABSF,      // d = |x|
    LDOBS,      // d = obs[x]
    LDPARAM,   // d = params[lane, x]
    LDCONST,   // d = consts[x]
    CKST,      // ckpt rows r .. r + n - 1 of this lane = registers a .. a + n - 1   (x = ck_field(r, n))
    CKLD,      // registers a .. a + n - 1 = ckpt rows r .. r + n - 1 of this lane   (x = ck_field(r, n))
    MSUB,      // d = x * y - z  (product rounded, then difference rounded)
    RSUB,      // d = z - x * y  (product rounded, then difference rounded)
    SKIP,      // skip the next n instructions (n = imm & kSkipCountMask) when every lane of the wave has
               // predicate register x == 0 (side bit clear: the then-arm follows) or every lane has it
               // nonzero (side bit set: the else-arm follows); the skipped arm's results are never read
    HOT_END,
    // ---- cold forms: sine and cosine (their library code branches per
    // lane), pow, and the loss and gradient stores (masked per slot)
    UN = 40,   // d = f(x), f = imm: see Unary
    POWF,      // d = pow(x, y)   (heavy: kept out of line to spare registers)
    STLOSS,    // loss[lane] = register a          (slots < imm only)
    STGRAD,    // grad[lane, x] = register a       (slots < imm only)
    END = 63,
};

enum Unary : uint32_t { U_SIN = 0, U_COS };

constexpr uint32_t kFormMask = 63u;
constexpr uint32_t kSkipSideShift = 17, kSkipCountMask = (1u << kSkipSideShift) - 1;
constexpr uint32_t kFirstShift = 6, kImmShift = 14;
constexpr uint32_t kMacBit = 1u << 10, kAccBit = 1u << 11, kMsubBit = 1u << 12, kBlockBit = 1u << 13;
// Order of the replay's bit tests ahead of its dispatch tree (chosen per
// launch from the programs' instruction counts; the first form tested runs
// without a taken branch): multiply-add then the linear adjoint rule; the
// adjoint rule, multiply-add and multiply-subtract; multiply-add then the
// block dots.
enum DispatchOrder : int { kOrderMacAcc = 0, kOrderAccMacMsub = 1, kOrderMacBlock = 2 };
// the form's own bits of a header (form number and its one-hot flag)
inline uint32_t form_bits(uint32_t form) {
    return form | (form == MAC ? kMacBit : 0u) | (form == ACC ? kAccBit : 0u) | (form == MSUB ? kMsubBit : 0u) |
           (form == DOTB || form == DOTBACC ? kBlockBit : 0u);
}
constexpr uint32_t kMaxImm = (1u << 18) - 1;
constexpr uint32_t kMaxBlock = 4;            // outputs of a block form (sink and trash rows reserved)

// Checkpoint moves (CKST, CKLD) carry their own row count per slot, up to
// kMaxCk rows, in the index field: x = row | (n - 1) << kCkRowBits; the
// header immediate is the largest count of the instruction's slots, and a
// slot with fewer rows repeats its last move (same register, same row, same
// value), so every slot runs the same uniform loop.  Slots an instruction
// does not use move one row between a sink register and a trash row.
constexpr uint32_t kMaxCk = 16;
constexpr uint32_t kCkRowBits = 28;
constexpr uint32_t kCkRowMask = (1u << kCkRowBits) - 1;
inline uint32_t ck_field(uint32_t row, uint32_t n) { return row | (n - 1) << kCkRowBits; }
inline bool is_ckmove(uint32_t form) { return form == CKST || form == CKLD; }

// immediates: DOT / DOTACC: K | negate << 5 | sa << 6 | sb << 12;
// DOTB / DOTBACC: K | N << 3 | sx << 6 | sy << 9 | sc << 12 | negate << 15
inline uint32_t dot_imm(uint32_t K, uint32_t sa, uint32_t sb, bool neg) {
    return K | uint32_t(neg) << 5 | sa << 6 | sb << 12;
}
inline uint32_t dotb_imm(uint32_t K, uint32_t N, uint32_t sx, uint32_t sy, uint32_t sc, bool neg) {
    return K | N << 3 | sx << 6 | sy << 9 | sc << 12 | uint32_t(neg) << 15;
}

// Program fetch: the slot words come in chunks of kChunk instructions as
// 4 rows x kChunk x 4 words; row r (threads 16r .. 16r + 15 of a wave)
// carries the micro-ops of slot r * S / 4, and thread 16r + j holds word j
// of its row (instruction j / 4, word j % 4), so one coalesced dword load per
// thread fetches the chunk and a row broadcast hands every thread of a slot
// its words.  The headers follow the chunks, kHeaderGroup at a time: thread
// t of a wave holds the four headers of chunk t of a group (one 16-byte
// load), so the four instructions of a chunk read their headers from one
// lane.  The chunk holding END is followed by two more chunks and the header
// group holding it by two more groups (the fetch reads two ahead).  Slot
// counts 1, 2 and 4 (a slot's threads fill whole rows).
constexpr uint32_t kChunk = 4;
constexpr uint32_t kRows = 4;
constexpr uint32_t kChunkWords = kRows * kChunk * 4;
constexpr uint32_t kFetchAhead = 2;
constexpr uint32_t kHeaderGroup = 64 * kChunk;
constexpr uint32_t kMaxSlots = 4;

inline bool is_hot(uint32_t form) { return form >= MAC && form < HOT_END; }
// forms whose register a is written
inline bool writes_a(uint32_t form) {
    return form != CKST && form != STLOSS && form != STGRAD && form != SKIP && form != END;
}
// forms whose field x is an index rather than a register
inline bool x_is_index(uint32_t form) {
    return form == LDOBS || form == LDPARAM || form == LDCONST || form == CKST || form == CKLD || form == STGRAD;
}

}  // namespace slot

// Per-program constants read by the kernel: the device program and where the
// program's checkpoint and spill rows start in the workspace.  Depends only
// on the program and the launch's register budget, never on per-call
// pointers, so a table of these can be cached on the device.
struct ProgStatic {
    const uint32_t *prog;    // slot words, chunk-major ([chunk][row][instr][4]), then the headers
    const double *consts;    // constant pool
    uint64_t ckpt_row0;      // checkpoint row r of lane l at ws[(ckpt_row0 + r)*Lpad + l]
    uint64_t spill_row0;     // register r_lds + r of lane l at ws[(spill_row0 + r)*Lpad + l]
    uint32_t hdr_off;        // word offset of the headers in prog
    uint32_t r_lds;          // registers held in LDS
    uint32_t spills;         // nonzero when the program has registers beyond r_lds
};

// Kernel variant of a launch: every register in LDS, a spill tail for every
// program, or chosen per program (many-program launches that mix the two).
enum LaunchVariant : int { kLdsOnly = 0, kSpill = 1, kPerProgram = 2 };

// Per-call arguments.  Program q of a launch (blockIdx.y) reads
// params + q*prog_stride_p and writes loss + q*L, grad + q*prog_stride_g.
// With n_points > 0 the data axis is flattened into the lanes: lane f serves
// parameter row f / n_points and data point f % n_points, whose observation
// row starts at obs + (f % n_points) * obs_stride; loss[f] and
// grad[f*ld_g + p] are then that point's term and term gradient.
struct LaunchArgs {
    const double *obs;
    const double *params;
    double *loss;
    double *grad;
    double *ws;
    int64_t ld_p, ld_g, L, Lpad, prog_stride_p, prog_stride_g;
    int64_t n_points = 0, obs_stride = 0;
    // Many-program launches laid out per XCD: a one-dimensional grid of n_wg
    // workgroups, workgroup w taking the work item wg_items[w] = program << 32
    // | lane block (all ones: none).  Null: program blockIdx.y, lane block
    // blockIdx.x.
    const uint64_t *wg_items = nullptr;
    uint32_t n_wg = 0;
};

}  // namespace ndvm
