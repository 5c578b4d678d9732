// Tape validation: serialized bytes -> Tape, rejecting anything the
// scheduler or the kernels could not handle safely (forward references,
// shape mismatches, out-of-range pool/param/obs/aux indices, nonzero unused
// fields).
#include <cstdio>

#include "common.h"

namespace ndvm {

namespace {
thread_local std::string g_error;

bool fail(const char *what, uint32_t k) {
    char m[160];
    std::snprintf(m, sizeof m, "invalid tape: %s (op %u)", what, k);
    set_error(m);
    return false;
}

bool check_op(const Tape &t, uint32_t k) {
    const TapeOp &o = t.ops[k];
    auto ref = [&](uint32_t s) { return s < k; };
    int r = 0, c = 0;
    switch (o.code) {
    case tp::CONST:
        if (o.rows != 1 || o.cols != 1 || o.imm >= t.consts.size() || o.a || o.b || o.c || o.d)
            return fail("bad CONST", k);
        return true;
    case tp::PARAM:
        if (o.rows != 1 || o.cols != 1 || o.imm >= t.n_params || o.a || o.b || o.c || o.d)
            return fail("bad PARAM", k);
        return true;
    case tp::OBS:
        if (o.rows != 1 || o.cols != 1 || o.imm >= t.n_obs || o.a || o.b || o.c || o.d)
            return fail("bad OBS", k);
        return true;
    case tp::PACK: {
        uint64_t n = uint64_t(o.rows) * o.cols;
        if (o.rows < 1 || o.rows > 4 || o.cols < 1 || o.cols > 4 || o.b != n || o.c || o.d || o.imm)
            return fail("bad PACK", k);
        if (uint64_t(o.a) + n > t.aux.size()) return fail("PACK list out of range", k);
        for (uint32_t i = 0; i < n; ++i) {
            uint32_t s = t.aux[o.a + i];
            if (!ref(s) || t.nel(s) != 1) return fail("bad PACK element", k);
        }
        return true;
    }
    case tp::INDEX:
        if (!ref(o.a) || o.rows != 1 || o.cols != 1 || o.imm >= t.nel(o.a) || o.b || o.c || o.d)
            return fail("bad INDEX", k);
        return true;
    case tp::SELECT:
        if (!ref(o.a) || !ref(o.b) || !ref(o.c) || !ref(o.d) || o.imm) return fail("bad SELECT", k);
        if (t.nel(o.a) != 1 || t.nel(o.b) != 1) return fail("SELECT predicate not scalar", k);
        if (t.ops[o.c].rows != o.rows || t.ops[o.c].cols != o.cols || t.ops[o.d].rows != o.rows ||
            t.ops[o.d].cols != o.cols)
            return fail("SELECT shape", k);
        return true;
    case tp::NEG: case tp::EXP: case tp::LOG: case tp::SQRT: case tp::SIN: case tp::COS:
    case tp::ABS: case tp::TRANSPOSE: case tp::TRACE: case tp::INV: case tp::DET: case tp::LOGDET:
        if (!ref(o.a) || o.b || o.c || o.d || o.imm) return fail("bad unary op", k);
        if (!op_shape(o.code, t.ops[o.a].rows, t.ops[o.a].cols, 0, 0, &r, &c) || r != o.rows || c != o.cols)
            return fail("unary shape", k);
        return true;
    case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: case tp::POW: case tp::DOT:
    case tp::MATMUL: case tp::OUTER:
        if (!ref(o.a) || !ref(o.b) || o.c || o.d || o.imm) return fail("bad binary op", k);
        if (!op_shape(o.code, t.ops[o.a].rows, t.ops[o.a].cols, t.ops[o.b].rows, t.ops[o.b].cols, &r, &c) ||
            r != o.rows || c != o.cols)
            return fail("binary shape", k);
        return true;
    }
    return fail("unknown opcode", k);
}

uint32_t rd32(const uint8_t *p) {
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}
}  // namespace

void set_error(const std::string &msg) { g_error = msg; }
const char *get_error() { return g_error.c_str(); }

ndvm_status parse_tape(const uint8_t *b, size_t n, Tape *out) {
    if (!b || n < kTapeHeaderBytes || std::memcmp(b, "NDVT", 4) != 0 || rd32(b + 4) != 1) {
        set_error("invalid tape: bad header");
        return NDVM_E_TAPE;
    }
    Tape &t = *out;
    t.n_params = rd32(b + 8);
    t.n_obs = rd32(b + 12);
    uint32_t n_ops = rd32(b + 16), n_consts = rd32(b + 20), n_aux = rd32(b + 24);
    t.loss = rd32(b + 28);
    uint64_t want = kTapeHeaderBytes + 8ull * n_consts + 4ull * n_aux + uint64_t(kTapeOpBytes) * n_ops;
    if (want != n || n_ops == 0 || n_ops > kMaxTapeOps) {
        set_error("invalid tape: size mismatch");
        return NDVM_E_TAPE;
    }
    const uint8_t *p = b + kTapeHeaderBytes;
    t.consts.resize(n_consts);
    std::memcpy(t.consts.data(), p, 8ull * n_consts);
    p += 8ull * n_consts;
    t.aux.resize(n_aux);
    std::memcpy(t.aux.data(), p, 4ull * n_aux);
    p += 4ull * n_aux;
    t.ops.resize(n_ops);
    for (uint32_t k = 0; k < n_ops; ++k, p += kTapeOpBytes) {
        TapeOp &o = t.ops[k];
        std::memcpy(&o.code, p, 2);
        o.rows = p[2];
        o.cols = p[3];
        o.a = rd32(p + 4);
        o.b = rd32(p + 8);
        o.c = rd32(p + 12);
        o.d = rd32(p + 16);
        o.imm = rd32(p + 20);
        if (o.rows < 1 || o.rows > 4 || o.cols < 1 || o.cols > 4) {
            fail("bad shape", k);
            return NDVM_E_TAPE;
        }
        if (!check_op(t, k)) return NDVM_E_TAPE;
    }
    if (t.loss >= n_ops || t.nel(t.loss) != 1) {
        set_error("invalid tape: loss slot");
        return NDVM_E_TAPE;
    }
    return NDVM_OK;
}

}  // namespace ndvm
