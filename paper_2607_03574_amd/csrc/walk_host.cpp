// Device walker, host side: validation and structural measurement of stack
// bytecode (no unrolling, no tape, no scheduling), packing of a program set
// into one device buffer, and the C-ABI entry points.  The walk itself runs
// on the GPU (walk.hip).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "common.h"
#include "walk.h"

namespace ndvm {
hipError_t launch_walk(const walk::Args &A, uint32_t grid, hipStream_t stream);
}

using namespace ndvm;

struct ndvm_walk {
    std::vector<walk::ProgDesc> descs;
    void *d_buf = nullptr;
    uint32_t n_prog = 0, n_obs = 0, max_params = 0;
    uint32_t n_nodes = 0, depth = 0, n_locals = 0, n_loops = 0, n_frames = 0;
    int device = 0;
    ~ndvm_walk() {
        if (d_buf) (void)hipFree(d_buf);
    }
};

namespace {

struct Fail {
    ndvm_status st;
    std::string msg;
};

[[noreturn]] void fail(ndvm_status st, const std::string &m) { throw Fail{st, m}; }

uint32_t rd32(const uint8_t *p) {
    uint32_t v;
    std::memcpy(&v, p, 4);
    return v;
}

struct Word {
    uint8_t op, a;
    uint16_t b;
    uint32_t imm;
};

bool scalar_unary(uint8_t op) {
    switch (op) {
    case bc::NEG: case bc::EXP: case bc::LOG: case bc::SQRT: case bc::SIN: case bc::COS: case bc::ABS:
        return true;
    }
    return false;
}
bool scalar_binary(uint8_t op) {
    switch (op) {
    case bc::ADD: case bc::SUB: case bc::MUL: case bc::DIV: case bc::POW:
        return true;
    }
    return false;
}
bool matrix_word(uint8_t op) {
    switch (op) {
    case bc::DOT: case bc::MATMUL: case bc::TRANSPOSE: case bc::INV: case bc::DET: case bc::LOGDET:
    case bc::TRACE: case bc::OUTER: case bc::PACK: case bc::INDEX:
        return true;
    }
    return false;
}

// operand stack words a (scalar) bytecode word pops and pushes
void stack_effect(uint8_t op, uint32_t *pops, uint32_t *pushes) {
    switch (op) {
    case bc::PUSH: case bc::OBS: case bc::PARAM: case bc::LOADL: *pops = 0; *pushes = 1; return;
    case bc::STOREL: case bc::DROP: *pops = 1; *pushes = 0; return;
    case bc::DUP: *pops = 1; *pushes = 2; return;
    case bc::OVER: *pops = 2; *pushes = 3; return;
    case bc::SWAP: *pops = 2; *pushes = 2; return;
    case bc::IFLT: *pops = 2; *pushes = 0; return;
    default:
        if (scalar_binary(op)) { *pops = 2; *pushes = 1; return; }
        if (scalar_unary(op)) { *pops = 1; *pushes = 1; return; }
        *pops = 0;   // HALT, LOOP, ENDLOOP, ELSE, ENDIF, OBSX
        *pushes = 0;
    }
}

// Structural measurement of one program: what one wave's walk can reach,
// found by following the block structure once (a loop body is measured at
// its first and last trip, whose entry depths bound every trip's).
class Measure {
  public:
    uint32_t n_params = 0, n_obs = 0, n_consts = 0;
    std::vector<Word> code;
    std::vector<int32_t> match;
    std::vector<double> consts;
    uint32_t n_locals = 0;

    // results
    uint64_t nodes = 0, steps = 0;
    int64_t max_depth = 0;
    uint32_t max_frames = 0, max_loops = 0;

    void load(const uint8_t *b, size_t n) {
        if (!b || n < 24 || std::memcmp(b, "NDVB", 4) != 0) fail(NDVM_E_BYTECODE, "bad NDVB header");
        if (rd32(b + 4) != 1) fail(NDVM_E_BYTECODE, "unsupported NDVB version");
        n_params = rd32(b + 8);
        n_obs = rd32(b + 12);
        const uint32_t ni = rd32(b + 16), nc = rd32(b + 20);
        if (24ull + 8ull * ni + 8ull * nc != n) fail(NDVM_E_BYTECODE, "NDVB size mismatch");
        code.resize(ni);
        for (uint32_t k = 0; k < ni; ++k) {
            const uint8_t *w = b + 24 + 8ull * k;
            code[k] = Word{w[0], w[1], uint16_t(w[2] | (w[3] << 8)), rd32(w + 4)};
        }
        consts.resize(nc);
        std::memcpy(consts.data(), b + 24 + 8ull * ni, 8ull * nc);
        n_consts = nc;
        pair_blocks();
        for (const Word &w : code)
            if (w.op == bc::LOADL || w.op == bc::STOREL) {
                if (w.imm >= walk::kMaxLocals) fail(NDVM_E_UNSUPPORTED, "local index beyond the device walker's limit");
                n_locals = std::max(n_locals, w.imm + 1);
            }
    }

    void pair_blocks() {
        match.assign(code.size(), -1);
        std::vector<int32_t> st;
        for (size_t pc = 0; pc < code.size(); ++pc) {
            const uint8_t op = code[pc].op;
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
                const uint32_t ns = code[pc].a;
                for (uint32_t d = 1; d <= ns; ++d)
                    if (pc + d >= code.size() || code[pc + d].op != bc::OBSX) fail(NDVM_E_BYTECODE, "missing OBSX word");
                pc += ns;
            }
        }
        if (!st.empty()) fail(NDVM_E_BYTECODE, "unterminated block");
    }

    struct State {
        int64_t depth = 0;
        std::vector<uint8_t> set;   // locals holding a value
    };

    // trips of the enclosing loops, outermost first
    std::vector<uint32_t> trips;

    static uint64_t sat_add(uint64_t a, uint64_t b) { return a + b < a ? ~0ull : a + b; }
    static uint64_t sat_mul(uint64_t a, uint64_t b) { return b && a > ~0ull / b ? ~0ull : a * b; }

    // Walk words [pc, stop) from state s; returns the nodes recorded.
    // Sets *halted when a HALT is met at the top level.
    uint64_t block(size_t pc, size_t stop, State &s, bool top, uint32_t frames, bool *halted, uint64_t *words) {
        uint64_t n = 0, wds = 0;
        struct Flush {
            uint64_t *out, *val;
            ~Flush() { *out = sat_add(*out, *val); }
        } flush{words, &wds};
        auto need = [&](int64_t k) {
            if (s.depth < k) fail(NDVM_E_BYTECODE, "stack underflow");
        };
        auto push = [&]() {
            ++s.depth;
            max_depth = std::max(max_depth, s.depth);
            if (s.depth > int64_t(walk::kMaxDepth)) fail(NDVM_E_UNSUPPORTED, "stack deeper than the device walker's limit");
        };
        while (pc < stop) {
            const Word w = code[pc];
            wds = sat_add(wds, 1);
            switch (w.op) {
            case bc::HALT:
                if (!top) fail(NDVM_E_BYTECODE, "HALT inside a block");
                if (s.depth != 1) fail(NDVM_E_BYTECODE, "HALT needs one scalar");
                *halted = true;
                return n;
            case bc::PUSH:
                if (w.imm >= n_consts) fail(NDVM_E_BYTECODE, "bad const index");
                push();
                n = sat_add(n, 1);
                break;
            case bc::PARAM:
                if (w.imm >= n_params) fail(NDVM_E_BYTECODE, "bad param index");
                push();
                break;
            case bc::OBS: {
                if (w.a > trips.size()) fail(NDVM_E_BYTECODE, "OBS stride beyond loop depth");
                int64_t lo = w.imm, hi = w.imm;
                for (uint32_t d = 0; d < w.a; ++d) {
                    int32_t stride;
                    const uint32_t raw = code[pc + 1 + d].imm;
                    std::memcpy(&stride, &raw, 4);
                    const int64_t span = int64_t(stride) * int64_t(trips[trips.size() - 1 - d] - 1);
                    if (span < 0) lo += span; else hi += span;
                }
                if (lo < 0 || hi >= int64_t(n_obs)) fail(NDVM_E_BYTECODE, "obs index out of range");
                push();
                n = sat_add(n, 1);
                pc += w.a;
                break;
            }
            case bc::OBSX:
                fail(NDVM_E_BYTECODE, "stray OBSX word");
            case bc::LOADL:
                if (w.imm >= s.set.size() || !s.set[w.imm]) fail(NDVM_E_BYTECODE, "unset local");
                push();
                break;
            case bc::STOREL:
                need(1);
                --s.depth;
                s.set[w.imm] = 1;
                break;
            case bc::DUP:
                need(1);
                push();
                break;
            case bc::OVER:
                need(2);
                push();
                break;
            case bc::SWAP:
                need(2);
                break;
            case bc::DROP:
                need(1);
                --s.depth;
                break;
            case bc::LOOP: {
                const size_t end = size_t(match[pc]);
                if (w.imm > 0) {
                    trips.push_back(w.imm);
                    if (trips.size() > walk::kMaxLoops) fail(NDVM_E_UNSUPPORTED, "loops nested beyond the device walker's limit");
                    max_loops = std::max<uint32_t>(max_loops, uint32_t(trips.size()));
                    // first trip from the entry state; its exit gives the depth change
                    State first = s;
                    bool h = false;
                    uint64_t wb = 0;
                    const uint64_t nb = block(pc + 1, end, first, false, frames, &h, &wb);
                    const int64_t delta = first.depth - s.depth;
                    uint64_t per = nb;
                    if (delta != 0 && w.imm > 1) {
                        // the last trip's entry depth bounds every trip's depth
                        // and merge count from the other side
                        State last = first;
                        last.depth = s.depth + delta * int64_t(w.imm - 1);
                        if (last.depth < 0) fail(NDVM_E_BYTECODE, "stack underflow");
                        State probe = last;
                        uint64_t wl = 0;
                        per = std::max(per, block(pc + 1, end, probe, false, frames, &h, &wl));
                        wb = std::max(wb, wl);
                    }
                    trips.pop_back();
                    n = sat_add(n, sat_mul(per, w.imm));
                    wds = sat_add(wds, sat_mul(wb + 1, w.imm));   // the body and its ENDLOOP, every trip
                    s.set = first.set;
                    s.depth += delta * int64_t(w.imm);
                    if (s.depth < 0) fail(NDVM_E_BYTECODE, "stack underflow");
                    max_depth = std::max(max_depth, s.depth);
                }
                pc = end;
                break;
            }
            case bc::IFLT: {
                const size_t els = size_t(match[pc]), end = size_t(match[els]);
                need(2);
                s.depth -= 2;
                if (frames + 1 > walk::kMaxFrames) fail(NDVM_E_UNSUPPORTED, "branches nested beyond the device walker's limit");
                max_frames = std::max(max_frames, frames + 1);
                State a = s, b = s;
                bool h = false;
                uint64_t wa = 0, wb = 0;
                const uint64_t na = block(pc + 1, els, a, false, frames + 1, &h, &wa);
                const uint64_t nb = block(els + 1, end, b, false, frames + 1, &h, &wb);
                wds = sat_add(wds, sat_add(sat_add(wa, wb), 2));   // both arms, ELSE and ENDIF
                if (a.depth != b.depth) fail(NDVM_E_STRUCT_DIVERGE, "branch arms leave different stack depths");
                if (a.set != b.set) fail(NDVM_E_STRUCT_DIVERGE, "a local is set in one branch arm only");
                // one merge per stack position and local at most
                n = sat_add(n, sat_add(sat_add(na, nb), uint64_t(a.depth) + n_locals));
                s = a;
                pc = end;
                break;
            }
            case bc::ELSE: case bc::ENDIF: case bc::ENDLOOP:
                fail(NDVM_E_BYTECODE, "unexpected block word");
            default:
                if (matrix_word(w.op)) fail(NDVM_E_UNSUPPORTED, "the device walker runs scalar programs only");
                if (scalar_unary(w.op)) {
                    need(1);
                } else if (scalar_binary(w.op)) {
                    need(2);
                    --s.depth;
                } else {
                    char m[64];
                    std::snprintf(m, sizeof m, "unknown opcode 0x%02x", w.op);
                    fail(NDVM_E_BYTECODE, m);
                }
                n = sat_add(n, 1);
            }
            ++pc;
        }
        if (top) fail(NDVM_E_BYTECODE, "missing HALT");
        return n;
    }

    void run() {
        State s;
        s.set.assign(n_locals, 0);
        bool halted = false;
        nodes = sat_add(block(0, code.size(), s, true, 0, &halted, &steps), n_params);
        if (nodes > walk::kMaxNodes) fail(NDVM_E_UNSUPPORTED, "program records more nodes than the device walker holds");
        if (steps >= 0xFFFFFFFFull) fail(NDVM_E_UNSUPPORTED, "program executes more words than the device walker counts");
        if (walk::lds_bytes(uint32_t(max_depth), n_locals, max_loops, max_frames, uint32_t(nodes), n_params) >
            walk::kMaxLdsBytes)
            fail(NDVM_E_UNSUPPORTED, "the walk's structural state exceeds a workgroup's LDS");
    }
};

template <class F>
ndvm_status guarded(F f) {
    try {
        return f();
    } catch (const Fail &e) {
        set_error(e.msg);
        return e.st;
    } catch (const std::bad_alloc &) {
        set_error("out of host memory");
        return NDVM_E_NOMEM;
    } catch (const std::exception &e) {
        set_error(std::string("internal error: ") + e.what());
        return NDVM_E_INTERNAL;
    }
}

constexpr uint32_t kStatusBytes = 256;   // status word, then the wave slots (256-byte aligned)

// Wave slots one launch uses: enough waves to fill every CU to the
// occupancy the LDS allows (at most 16 per CU), never more than the work.
uint32_t wave_slots(const ndvm_walk &w, uint64_t items) {
    int dev = 0, cus = 256, lds = 160 * 1024;
    if (hipGetDevice(&dev) == hipSuccess) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) cus = v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) == hipSuccess && v > 0)
            lds = v;
    }
    const uint64_t lds_wave = walk::lds_bytes(w.depth, w.n_locals, w.n_loops, w.n_frames, w.n_nodes, w.max_params);
    const uint64_t per_cu = std::max<uint64_t>(1, std::min<uint64_t>(16, uint64_t(lds) / std::max<uint64_t>(lds_wave, 1)));
    return uint32_t(std::min<uint64_t>(items, per_cu * uint64_t(cus)));
}

}  // namespace

extern "C" {

ndvm_status ndvm_walk_prepare(const uint8_t *const *bytecodes, const size_t *lens, int n_prog, void *stream,
                              ndvm_walk **out) {
    return guarded([&]() -> ndvm_status {
        if (!bytecodes || !lens || !out || n_prog <= 0) {
            set_error("ndvm_walk_prepare: null argument or no program");
            return NDVM_E_ARG;
        }
        auto w = std::make_unique<ndvm_walk>();
        w->n_prog = uint32_t(n_prog);
        std::vector<Measure> ms(static_cast<size_t>(n_prog));
        for (int q = 0; q < n_prog; ++q) {
            Measure &m = ms[size_t(q)];
            try {
                m.load(bytecodes[q], lens[q]);
                m.run();
            } catch (Fail &e) {
                e.msg = "program " + std::to_string(q) + ": " + e.msg;
                throw;
            }
            if (q > 0 && m.n_obs != w->n_obs) fail(NDVM_E_ARG, "ndvm_walk_prepare: programs read different observation counts");
            w->n_obs = m.n_obs;
        }
        // device buffer: descriptors, then per program its code, matches and
        // constants (doubles 8-byte aligned)
        const uint32_t desc_words = uint32_t(sizeof(walk::ProgDesc) / 4) * uint32_t(n_prog);
        std::vector<uint32_t> buf(desc_words, 0);
        w->descs.resize(size_t(n_prog));
        for (int q = 0; q < n_prog; ++q) {
            const Measure &m = ms[size_t(q)];
            walk::ProgDesc &d = w->descs[size_t(q)];
            d.n_instr = uint32_t(m.code.size());
            d.n_params = m.n_params;
            d.n_obs = m.n_obs;
            d.n_nodes = uint32_t(std::max<uint64_t>(m.nodes, 1));
            d.depth = uint32_t(std::max<int64_t>(m.max_depth, 1));
            d.n_locals = m.n_locals;
            d.n_frames = m.max_frames;
            d.n_loops = m.max_loops;
            d.n_steps = uint32_t(m.steps);
            d.code_off = uint32_t(buf.size());
            for (const Word &x : m.code) {
                uint32_t pops = 0, pushes = 0;
                stack_effect(x.op, &pops, &pushes);
                buf.push_back(uint32_t(x.op) | uint32_t(x.a) << 8 | pops << 16 | pushes << 18);
                buf.push_back(x.imm);
            }
            d.match_off = uint32_t(buf.size());
            for (int32_t v : m.match) buf.push_back(uint32_t(v));
            if (buf.size() % 2) buf.push_back(0);
            d.const_off = uint32_t(buf.size());
            for (double c : m.consts) {
                uint32_t two[2];
                std::memcpy(two, &c, 8);
                buf.push_back(two[0]);
                buf.push_back(two[1]);
            }
            w->max_params = std::max(w->max_params, d.n_params);
            w->n_nodes = std::max(w->n_nodes, d.n_nodes);
            w->depth = std::max(w->depth, d.depth);
            w->n_locals = std::max(w->n_locals, d.n_locals);
            w->n_loops = std::max(w->n_loops, d.n_loops);
            w->n_frames = std::max(w->n_frames, d.n_frames);
        }
        if (buf.size() > 0xFFFFFFFFull) fail(NDVM_E_UNSUPPORTED, "program set beyond the device buffer's 32-bit offsets");
        if (walk::lds_bytes(w->depth, w->n_locals, w->n_loops, w->n_frames, w->n_nodes, w->max_params) >
            walk::kMaxLdsBytes)
            fail(NDVM_E_UNSUPPORTED, "the program set's structural state exceeds a workgroup's LDS");
        std::memcpy(buf.data(), w->descs.data(), sizeof(walk::ProgDesc) * size_t(n_prog));
        if (hipGetDevice(&w->device) != hipSuccess) {
            set_error("hipGetDevice failed");
            return NDVM_E_DEVICE;
        }
        if (hipMalloc(&w->d_buf, buf.size() * 4) != hipSuccess) {
            (void)hipGetLastError();
            w->d_buf = nullptr;
            set_error("hipMalloc of the walker's program buffer failed");
            return NDVM_E_NOMEM;
        }
        const hipStream_t s = static_cast<hipStream_t>(stream);
        if (hipMemcpyAsync(w->d_buf, buf.data(), buf.size() * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) {
            set_error("copy of the walker's program buffer failed");
            return NDVM_E_DEVICE;
        }
        *out = w.release();
        return NDVM_OK;
    });
}

ndvm_status ndvm_walk_measure(const uint8_t *bytecode, size_t len, ndvm_walk_info *out) {
    return guarded([&]() -> ndvm_status {
        if (!bytecode || !out) {
            set_error("ndvm_walk_measure: null argument");
            return NDVM_E_ARG;
        }
        Measure m;
        m.load(bytecode, len);
        m.run();
        out->n_params = m.n_params;
        out->n_obs = m.n_obs;
        out->n_nodes = m.nodes;
        out->depth = uint32_t(m.max_depth);
        out->n_locals = m.n_locals;
        out->n_frames = m.max_frames;
        out->n_loops = m.max_loops;
        return NDVM_OK;
    });
}

ndvm_status ndvm_walk_workspace_bytes(const ndvm_walk *w, int64_t L, size_t *bytes) {
    return guarded([&]() -> ndvm_status {
        if (!w || !bytes || L < 0) {
            set_error("ndvm_walk_workspace_bytes: null argument or negative L");
            return NDVM_E_ARG;
        }
        const uint64_t items = uint64_t(w->n_prog) * uint64_t((L + 63) / 64);
        const uint64_t slots = items ? wave_slots(*w, items) : 0;
        *bytes = size_t(kStatusBytes + slots * uint64_t(w->n_nodes) * walk::ws_bytes_per_node());
        return NDVM_OK;
    });
}

ndvm_status ndvm_walk_grad(const ndvm_walk *w, const double *params, int64_t L, int64_t ld_p, int64_t prog_stride_p,
                           const double *obs, int64_t n_obs, double *loss, double *grad, int64_t ld_g,
                           int64_t prog_stride_g, void *workspace, size_t workspace_bytes, void *stream) {
    return guarded([&]() -> ndvm_status {
        if (!w || L < 0 || (L > 0 && (!params || !loss || !grad || !workspace)) || (n_obs > 0 && !obs)) {
            set_error("ndvm_walk_grad: null argument or negative L");
            return NDVM_E_ARG;
        }
        if (n_obs != int64_t(w->n_obs)) {
            set_error("ndvm_walk_grad: n_obs differs from the programs' observation count");
            return NDVM_E_ARG;
        }
        if (ld_p < int64_t(w->max_params) || ld_g < int64_t(w->max_params) ||
            (w->n_prog > 1 && (prog_stride_p < L * ld_p || prog_stride_g < L * ld_g))) {
            set_error("ndvm_walk_grad: leading dimension or program stride too small");
            return NDVM_E_ARG;
        }
        if (L == 0) return NDVM_OK;
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev != w->device) {
            set_error("ndvm_walk_grad: the program set was prepared on another device");
            return NDVM_E_ARG;
        }
        size_t need = 0;
        ndvm_status st = ndvm_walk_workspace_bytes(w, L, &need);
        if (st != NDVM_OK) return st;
        if (workspace_bytes < need) {
            set_error("ndvm_walk_grad: workspace too small (see ndvm_walk_workspace_bytes)");
            return NDVM_E_NOMEM;
        }
        walk::Args A{};
        A.buf = static_cast<const uint32_t *>(w->d_buf);
        A.n_prog = w->n_prog;
        A.L = L;
        A.params = params;
        A.ld_p = ld_p;
        A.prog_stride_p = prog_stride_p;
        A.obs = obs;
        A.loss = loss;
        A.grad = grad;
        A.ld_g = ld_g;
        A.prog_stride_g = prog_stride_g;
        A.ws = static_cast<uint8_t *>(workspace) + kStatusBytes;
        A.n_nodes_max = w->n_nodes;
        A.depth = w->depth;
        A.n_locals = w->n_locals;
        A.n_loops = w->n_loops;
        A.n_frames = w->n_frames;
        A.n_params = w->max_params;
        A.lds_bytes = uint32_t(walk::lds_bytes(w->depth, w->n_locals, w->n_loops, w->n_frames, w->n_nodes, w->max_params));
        A.n_items = uint64_t(w->n_prog) * uint64_t((L + 63) / 64);
        A.status = static_cast<int *>(workspace);
        const hipStream_t s = static_cast<hipStream_t>(stream);
        if (hipMemsetAsync(workspace, 0, sizeof(int), s) != hipSuccess) {
            set_error("ndvm_walk_grad: clearing the status word failed");
            return NDVM_E_DEVICE;
        }
        const hipError_t e = launch_walk(A, wave_slots(*w, A.n_items), s);
        if (e != hipSuccess) {
            set_error(std::string("walker launch failed: ") + hipGetErrorString(e));
            return NDVM_E_DEVICE;
        }
        return NDVM_OK;
    });
}

ndvm_status ndvm_walk_status(const void *workspace, void *stream) {
    return guarded([&]() -> ndvm_status {
        if (!workspace) {
            set_error("ndvm_walk_status: null workspace");
            return NDVM_E_ARG;
        }
        int code = 0;
        const hipStream_t s = static_cast<hipStream_t>(stream);
        if (hipMemcpyAsync(&code, workspace, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) {
            set_error("ndvm_walk_status: reading the status word failed");
            return NDVM_E_DEVICE;
        }
        if (code != 0) {
            set_error("the device walk met a bound its validation should have excluded (code " + std::to_string(code) +
                      "); the affected lanes hold NaN");
            return NDVM_E_INTERNAL;
        }
        return NDVM_OK;
    });
}

void ndvm_walk_free(ndvm_walk *w) { delete w; }

}  // extern "C"
