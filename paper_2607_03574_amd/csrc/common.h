// Internal definitions shared by the host parts of libndvm (trace producer,
// tape validator, scheduler, C ABI).  Not part of the public interface.
#pragma once

#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/ndvm.h"

namespace ndvm {

// ---- stack bytecode (NDVB) word opcodes ----
namespace bc {
enum : uint8_t {
    HALT = 0x00, PUSH = 0x01, PARAM = 0x02, OBS = 0x03, OBSX = 0x04,
    LOADL = 0x05, STOREL = 0x06, DUP = 0x07, SWAP = 0x08, DROP = 0x09, OVER = 0x0A,
    ADD = 0x10, SUB = 0x11, MUL = 0x12, DIV = 0x13, NEG = 0x14,
    EXP = 0x18, LOG = 0x19, SQRT = 0x1A, SIN = 0x1B, COS = 0x1C, POW = 0x1D, ABS = 0x1E,
    DOT = 0x20, MATMUL = 0x21, TRANSPOSE = 0x22, INV = 0x23, DET = 0x24, LOGDET = 0x25,
    TRACE = 0x26, OUTER = 0x27, PACK = 0x28, INDEX = 0x29,
    LOOP = 0x30, ENDLOOP = 0x31, IFLT = 0x32, ELSE = 0x33, ENDIF = 0x34,
};
}  // namespace bc

// ---- tape op codes: numeric words keep their bytecode numbers ----
namespace tp {
enum : uint16_t {
    CONST = 0x01, PARAM = 0x02, OBS = 0x03,
    ADD = 0x10, SUB = 0x11, MUL = 0x12, DIV = 0x13, NEG = 0x14,
    EXP = 0x18, LOG = 0x19, SQRT = 0x1A, SIN = 0x1B, COS = 0x1C, POW = 0x1D, ABS = 0x1E,
    DOT = 0x20, MATMUL = 0x21, TRANSPOSE = 0x22, INV = 0x23, DET = 0x24, LOGDET = 0x25,
    TRACE = 0x26, OUTER = 0x27, PACK = 0x28, INDEX = 0x29,
    SELECT = 0x40,
};
}  // namespace tp

constexpr uint32_t kMaxTapeOps = 1u << 26;
constexpr uint32_t kTapeHeaderBytes = 32;
constexpr uint32_t kTapeOpBytes = 24;

struct TapeOp {
    uint16_t code;
    uint8_t rows, cols;
    uint32_t a, b, c, d, imm;
};

struct Tape {
    uint32_t n_params = 0, n_obs = 0, loss = 0;
    std::vector<double> consts;
    std::vector<uint32_t> aux;
    std::vector<TapeOp> ops;
    uint32_t nel(uint32_t s) const { return uint32_t(ops[s].rows) * ops[s].cols; }
};

// Thread-local error message behind ndvm_last_error().
void set_error(const std::string &msg);
const char *get_error();

// Output shape of a numeric tape op from its operand shapes; false if invalid.
bool op_shape(uint16_t code, int ra, int ca, int rb, int cb, int *r, int *c);

// Trace producer: bytecode -> serialized tape bytes.
ndvm_status build_tape(const uint8_t *bc, size_t n, std::vector<uint8_t> *out);
// Validate serialized tape bytes into a Tape.
ndvm_status parse_tape(const uint8_t *bytes, size_t n, Tape *out);

}  // namespace ndvm
