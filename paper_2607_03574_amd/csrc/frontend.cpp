// Trace producer: one symbolic walk of a stack-bytecode program -> a
// lane-invariant tape.
//
// The walk carries slot ids and shapes, never numbers.  Each numeric word
// appends one tape op defining a fresh write-once slot (Section 3.4: tape
// nodes only for numeric primitives; structural words record nothing).
// Counted loops are unrolled here because their trip counts are structural
// (Section 3.3).  A numeric IFLT traces both arms from the same symbolic
// state and merges every stack position and local the arms left different
// with a per-lane SELECT (Section 6, lane-masked divergent control; the
// predicate carries no gradient, Property 1).  Arms that leave different
// stack depths, shapes or local sets are structural divergence and fail.
// An IFLT whose operands are both constant slots is resolved on the host.
#include <cmath>
#include <cstdio>
#include <map>

#include "common.h"

namespace ndvm {

namespace {

struct Word {
    uint8_t op, a;
    uint16_t b;
    uint32_t imm;
};

struct Err {
    ndvm_status st;
    std::string msg;
};

uint32_t rd32(const uint8_t *p) {
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}

class Tracer {
  public:
    uint32_t n_params = 0, n_obs = 0;
    std::vector<Word> code;
    std::vector<uint64_t> cbits;
    std::vector<int32_t> match;     // LOOP->ENDLOOP, IFLT->ELSE, ELSE->ENDIF
    std::vector<TapeOp> ops;
    std::vector<uint32_t> aux;
    std::vector<uint64_t> pool;     // tape const pool (bit patterns)
    std::vector<int32_t> pool_of;   // bytecode const index -> tape pool index
    std::vector<uint32_t> pool_src; // tape pool index -> bytecode const index
    std::vector<uint32_t> counters; // loop counters, outermost first

    void fail(ndvm_status st, const std::string &m) { throw Err{st, m}; }

    void load(const uint8_t *b, size_t n) {
        if (n < 24 || std::memcmp(b, "NDVB", 4) != 0) fail(NDVM_E_BYTECODE, "bad NDVB header");
        if (rd32(b + 4) != 1) fail(NDVM_E_BYTECODE, "unsupported NDVB version");
        n_params = rd32(b + 8);
        n_obs = rd32(b + 12);
        uint32_t ni = rd32(b + 16), nc = rd32(b + 20);
        if (24ull + 8ull * ni + 8ull * nc != n) fail(NDVM_E_BYTECODE, "NDVB size mismatch");
        code.resize(ni);
        for (uint32_t k = 0; k < ni; ++k) {
            const uint8_t *w = b + 24 + 8ull * k;
            code[k].op = w[0];
            code[k].a = w[1];
            code[k].b = uint16_t(w[2] | (w[3] << 8));
            code[k].imm = rd32(w + 4);
        }
        cbits.resize(nc);
        std::memcpy(cbits.data(), b + 24 + 8ull * ni, 8ull * nc);
        pool_of.assign(nc, -1);
        pair_blocks();
    }

    void pair_blocks() {
        match.assign(code.size(), -1);
        std::vector<int32_t> st;
        for (size_t pc = 0; pc < code.size(); ++pc) {
            uint8_t op = code[pc].op;
            if (op == bc::LOOP || op == bc::IFLT) {
                st.push_back(int32_t(pc));
            } else if (op == bc::ELSE) {
                if (st.empty() || code[st.back()].op != bc::IFLT) fail(NDVM_E_BYTECODE, "ELSE without IFLT");
                match[st.back()] = int32_t(pc);
                st.back() = int32_t(pc);
            } else if (op == bc::ENDIF) {
                if (st.empty() || code[st.back()].op != bc::ELSE) fail(NDVM_E_BYTECODE, "ENDIF without ELSE");
                match[st.back()] = int32_t(pc);
                st.pop_back();
            } else if (op == bc::ENDLOOP) {
                if (st.empty() || code[st.back()].op != bc::LOOP) fail(NDVM_E_BYTECODE, "ENDLOOP without LOOP");
                match[st.back()] = int32_t(pc);
                st.pop_back();
            } else if (op == bc::OBS) {
                uint32_t ns = code[pc].a;
                for (uint32_t d = 1; d <= ns; ++d)
                    if (pc + d >= code.size() || code[pc + d].op != bc::OBSX)
                        fail(NDVM_E_BYTECODE, "missing OBSX word");
                pc += ns;
            }
        }
        if (!st.empty()) fail(NDVM_E_BYTECODE, "unterminated block");
    }

    uint32_t emit(uint16_t code_, int r, int c, uint32_t a = 0, uint32_t b = 0, uint32_t cc = 0,
                  uint32_t d = 0, uint32_t imm = 0) {
        if (ops.size() >= kMaxTapeOps) fail(NDVM_E_BYTECODE, "tape too large");
        ops.push_back(TapeOp{code_, uint8_t(r), uint8_t(c), a, b, cc, d, imm});
        return uint32_t(ops.size() - 1);
    }

    int rows(uint32_t s) const { return ops[s].rows; }
    int cols(uint32_t s) const { return ops[s].cols; }
    bool scalar(uint32_t s) const { return ops[s].rows == 1 && ops[s].cols == 1; }

    std::vector<uint32_t> pop(std::vector<uint32_t> &st, size_t n) {
        if (st.size() < n) fail(NDVM_E_BYTECODE, "stack underflow");
        std::vector<uint32_t> out(st.end() - n, st.end());
        st.resize(st.size() - n);
        return out;
    }

    static bool is_unary(uint8_t op) {
        switch (op) {
        case bc::NEG: case bc::EXP: case bc::LOG: case bc::SQRT: case bc::SIN: case bc::COS:
        case bc::ABS: case bc::TRANSPOSE: case bc::TRACE: case bc::INV: case bc::DET:
        case bc::LOGDET:
            return true;
        }
        return false;
    }
    static bool is_binary(uint8_t op) {
        switch (op) {
        case bc::ADD: case bc::SUB: case bc::MUL: case bc::DIV: case bc::POW: case bc::DOT:
        case bc::MATMUL: case bc::OUTER:
            return true;
        }
        return false;
    }

    // Trace words [pc, stop).  Returns the loss slot at HALT (top level).
    int64_t block(size_t pc, size_t stop, std::vector<uint32_t> &st, std::map<uint32_t, uint32_t> &loc,
                  bool top, int depth) {
        if (depth > 512) fail(NDVM_E_BYTECODE, "blocks nested too deeply");
        while (pc < stop) {
            const Word w = code[pc];
            switch (w.op) {
            case bc::HALT:
                if (!top) fail(NDVM_E_BYTECODE, "HALT inside a block");
                if (st.size() != 1 || !scalar(st[0])) fail(NDVM_E_BYTECODE, "HALT needs one scalar");
                return st[0];
            case bc::PUSH: {
                if (w.imm >= cbits.size()) fail(NDVM_E_BYTECODE, "bad const index");
                if (pool_of[w.imm] < 0) {
                    pool_of[w.imm] = int32_t(pool.size());
                    pool.push_back(cbits[w.imm]);
                    pool_src.push_back(w.imm);
                }
                st.push_back(emit(tp::CONST, 1, 1, 0, 0, 0, 0, uint32_t(pool_of[w.imm])));
                break;
            }
            case bc::PARAM:
                if (w.imm >= n_params) fail(NDVM_E_BYTECODE, "bad param index");
                st.push_back(emit(tp::PARAM, 1, 1, 0, 0, 0, 0, w.imm));
                break;
            case bc::OBS: {
                if (w.a > counters.size()) fail(NDVM_E_BYTECODE, "OBS stride beyond loop depth");
                int64_t idx = w.imm;
                for (uint32_t d = 0; d < w.a; ++d) {
                    int32_t stride;
                    uint32_t raw = code[pc + 1 + d].imm;
                    std::memcpy(&stride, &raw, 4);
                    idx += int64_t(stride) * counters[counters.size() - 1 - d];
                }
                if (idx < 0 || idx >= int64_t(n_obs)) fail(NDVM_E_BYTECODE, "obs index out of range");
                st.push_back(emit(tp::OBS, 1, 1, 0, 0, 0, 0, uint32_t(idx)));
                pc += w.a;
                break;
            }
            case bc::OBSX:
                fail(NDVM_E_BYTECODE, "stray OBSX word");
                break;
            case bc::LOADL: {
                auto it = loc.find(w.imm);
                if (it == loc.end()) fail(NDVM_E_BYTECODE, "unset local");
                st.push_back(it->second);
                break;
            }
            case bc::STOREL:
                loc[w.imm] = pop(st, 1)[0];
                break;
            case bc::DUP: {
                uint32_t x = pop(st, 1)[0];
                st.push_back(x);
                st.push_back(x);
                break;
            }
            case bc::OVER: {
                auto v = pop(st, 2);
                st.push_back(v[0]);
                st.push_back(v[1]);
                st.push_back(v[0]);
                break;
            }
            case bc::SWAP: {
                auto v = pop(st, 2);
                st.push_back(v[1]);
                st.push_back(v[0]);
                break;
            }
            case bc::DROP:
                pop(st, 1);
                break;
            case bc::PACK: {
                int r = w.a, c = w.b;
                if (r < 1 || r > 4 || c < 1 || c > 4) fail(NDVM_E_BYTECODE, "bad PACK shape");
                auto els = pop(st, size_t(r) * c);
                for (uint32_t s : els)
                    if (!scalar(s)) fail(NDVM_E_BYTECODE, "PACK of a non-scalar");
                uint32_t off = uint32_t(aux.size());
                aux.insert(aux.end(), els.begin(), els.end());
                st.push_back(emit(tp::PACK, r, c, off, uint32_t(r * c)));
                break;
            }
            case bc::INDEX: {
                uint32_t s = pop(st, 1)[0];
                if (w.a >= rows(s) || w.b >= cols(s)) fail(NDVM_E_BYTECODE, "INDEX out of range");
                st.push_back(emit(tp::INDEX, 1, 1, s, 0, 0, 0, uint32_t(w.a * cols(s) + w.b)));
                break;
            }
            case bc::LOOP: {
                size_t end = size_t(match[pc]);
                counters.push_back(0);
                for (uint32_t k = 0; k < w.imm; ++k) {
                    counters.back() = k;
                    block(pc + 1, end, st, loc, false, depth + 1);
                }
                counters.pop_back();
                pc = end;
                break;
            }
            case bc::IFLT: {
                size_t els = size_t(match[pc]), end = size_t(match[els]);
                auto pr = pop(st, 2);
                uint32_t xa = pr[0], xb = pr[1];
                if (!scalar(xa) || !scalar(xb)) fail(NDVM_E_BYTECODE, "IFLT on a non-scalar");
                if (ops[xa].code == tp::CONST && ops[xb].code == tp::CONST) {
                    double va, vb;
                    std::memcpy(&va, &pool[ops[xa].imm], 8);
                    std::memcpy(&vb, &pool[ops[xb].imm], 8);
                    if (va < vb)
                        block(pc + 1, els, st, loc, false, depth + 1);
                    else
                        block(els + 1, end, st, loc, false, depth + 1);
                } else {
                    std::vector<uint32_t> s0 = st;
                    std::map<uint32_t, uint32_t> l0 = loc;
                    block(pc + 1, els, st, loc, false, depth + 1);
                    std::vector<uint32_t> s1 = st;
                    std::map<uint32_t, uint32_t> l1 = loc;
                    st = s0;
                    loc = l0;
                    block(els + 1, end, st, loc, false, depth + 1);
                    std::vector<uint32_t> s2 = st;
                    std::map<uint32_t, uint32_t> l2 = loc;
                    if (s1.size() != s2.size())
                        fail(NDVM_E_STRUCT_DIVERGE, "branch arms leave different stack depths");
                    for (size_t i = 0; i < s1.size(); ++i) {
                        uint32_t x = s1[i], y = s2[i];
                        if (rows(x) != rows(y) || cols(x) != cols(y))
                            fail(NDVM_E_STRUCT_DIVERGE, "branch arms leave different shapes");
                        st[i] = x == y ? x : emit(tp::SELECT, rows(x), cols(x), xa, xb, x, y);
                    }
                    std::map<uint32_t, uint32_t> merged;
                    auto i1 = l1.begin(), i2 = l2.begin();
                    while (i1 != l1.end() || i2 != l2.end()) {
                        if (i1 == l1.end() || i2 == l2.end() || i1->first != i2->first)
                            fail(NDVM_E_STRUCT_DIVERGE, "a local is set in one branch arm only");
                        uint32_t x = i1->second, y = i2->second;
                        if (rows(x) != rows(y) || cols(x) != cols(y))
                            fail(NDVM_E_STRUCT_DIVERGE, "branch arms leave different shapes");
                        merged[i1->first] = x == y ? x : emit(tp::SELECT, rows(x), cols(x), xa, xb, x, y);
                        ++i1;
                        ++i2;
                    }
                    loc = merged;
                }
                pc = end;
                break;
            }
            case bc::ELSE: case bc::ENDIF: case bc::ENDLOOP:
                fail(NDVM_E_BYTECODE, "unexpected block word");
                break;
            default: {
                if (!is_unary(w.op) && !is_binary(w.op)) {
                    char m[64];
                    std::snprintf(m, sizeof m, "unknown opcode 0x%02x", w.op);
                    fail(NDVM_E_BYTECODE, m);
                }
                bool bin = is_binary(w.op);
                auto v = pop(st, bin ? 2 : 1);
                int r, c;
                if (!op_shape(w.op, rows(v[0]), cols(v[0]), bin ? rows(v[1]) : 0, bin ? cols(v[1]) : 0, &r, &c))
                    fail(NDVM_E_BYTECODE, "shape error");
                st.push_back(emit(w.op, r, c, v[0], bin ? v[1] : 0));
            }
            }
            ++pc;
        }
        if (top) fail(NDVM_E_BYTECODE, "missing HALT");
        return -1;
    }
};

void put32(std::vector<uint8_t> &o, uint32_t v) {
    uint8_t b[4];
    std::memcpy(b, &v, 4);
    o.insert(o.end(), b, b + 4);
}

}  // namespace

bool op_shape(uint16_t code, int ra, int ca, int rb, int cb, int *r, int *c) {
    bool same = ra == rb && ca == cb;
    switch (code) {
    case tp::ADD: case tp::SUB:
        if (!same) return false;
        *r = ra; *c = ca;
        return true;
    case tp::MUL:
        if (same || (rb == 1 && cb == 1)) { *r = ra; *c = ca; return true; }
        if (ra == 1 && ca == 1) { *r = rb; *c = cb; return true; }
        return false;
    case tp::DIV:
        if (same || (rb == 1 && cb == 1)) { *r = ra; *c = ca; return true; }
        return false;
    case tp::NEG: case tp::EXP: case tp::LOG: case tp::SQRT: case tp::SIN: case tp::COS: case tp::ABS:
        *r = ra; *c = ca;
        return true;
    case tp::POW:
        if (ra != 1 || ca != 1 || rb != 1 || cb != 1) return false;
        *r = *c = 1;
        return true;
    case tp::DOT:
        if (!same) return false;
        *r = *c = 1;
        return true;
    case tp::MATMUL:
        if (ca != rb) return false;
        *r = ra; *c = cb;
        return true;
    case tp::TRANSPOSE:
        *r = ca; *c = ra;
        return true;
    case tp::TRACE:
        if (ra != ca) return false;
        *r = *c = 1;
        return true;
    case tp::INV:
        if (ra != ca || (ra != 1 && ra != 2)) return false;
        *r = ra; *c = ca;
        return true;
    case tp::DET: case tp::LOGDET:
        if (ra != ca || (ra != 1 && ra != 2)) return false;
        *r = *c = 1;
        return true;
    case tp::OUTER:
        if (ca != 1 || cb != 1) return false;
        *r = ra; *c = rb;
        return true;
    }
    return false;
}

ndvm_status build_tape(const uint8_t *b, size_t n, std::vector<uint8_t> *out) {
    Tracer T;
    int64_t loss;
    try {
        T.load(b, n);
        std::vector<uint32_t> st;
        std::map<uint32_t, uint32_t> loc;
        loss = T.block(0, T.code.size(), st, loc, true, 0);
    } catch (const Err &e) {
        set_error(e.msg);
        return e.st;
    } catch (const std::bad_alloc &) {
        set_error("out of host memory while tracing");
        return NDVM_E_NOMEM;
    }
    std::vector<uint8_t> &o = *out;
    o.clear();
    o.reserve(kTapeHeaderBytes + 8 * T.pool.size() + 4 * T.aux.size() + kTapeOpBytes * T.ops.size());
    o.insert(o.end(), {'N', 'D', 'V', 'T'});
    put32(o, 1);
    put32(o, T.n_params);
    put32(o, T.n_obs);
    put32(o, uint32_t(T.ops.size()));
    put32(o, uint32_t(T.pool.size()));
    put32(o, uint32_t(T.aux.size()));
    put32(o, uint32_t(loss));
    for (uint64_t v : T.pool) {
        uint8_t x[8];
        std::memcpy(x, &v, 8);
        o.insert(o.end(), x, x + 8);
    }
    for (uint32_t v : T.aux) put32(o, v);
    for (const TapeOp &op : T.ops) {
        uint8_t x[24];
        std::memcpy(x, &op.code, 2);
        x[2] = op.rows;
        x[3] = op.cols;
        std::memcpy(x + 4, &op.a, 4);
        std::memcpy(x + 8, &op.b, 4);
        std::memcpy(x + 12, &op.c, 4);
        std::memcpy(x + 16, &op.d, 4);
        std::memcpy(x + 20, &op.imm, 4);
        o.insert(o.end(), x, x + 24);
    }
    return NDVM_OK;
}

}  // namespace ndvm
