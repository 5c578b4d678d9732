// Tape scheduler.
//
// The tape is replayed by one GPU thread per lane.  This file decides, once
// per program and independently of L, where every lane value lives and what
// the reverse sweep recomputes:
//
//  * liveness (ops that cannot reach the loss are dropped) and activity
//    (values that do not depend on any parameter get no adjoint);
//  * checkpoint segments: the tape is cut where few values cross the cut;
//    the forward sweep stores the values a later segment needs at each cut,
//    the reverse sweep restores them, recomputes inside the segment only what
//    the segment's adjoint rules read, and applies the rules in reverse
//    order (Section 3.4 replay; the save policy is this build's own choice);
//  * values needed in many segments (loop invariants) stay resident instead
//    of being checkpointed at every cut;
//  * register allocation of values and adjoints on the instruction timeline
//    (first fit, contiguous blocks for matrices), separately for the forward
//    and the reverse phase;
//  * first-contribution flags, so adjoint registers need no zeroing: the
//    first write of an adjoint stores, later ones accumulate.
#include "sched.h"

#include <algorithm>
#include <map>
#include <unordered_map>

#include "isa.h"

namespace ndvm {

namespace {

enum Kind : uint8_t { K_COMP = 0, K_CONST = 1, K_OBS = 2, K_PARAM = 3 };

struct Info {
    const Tape &t;
    uint32_t N, P;
    std::vector<uint8_t> kind, nel, live, active, has_adj, need_rev;
    // Value numbering: rep[k] is the first slot that computes the same value
    // as slot k (same opcode, shape and immediate on the same operand values;
    // every op is a deterministic function of its operands, so the bits are
    // equal).  Only representatives are computed; every reader of a value
    // reads its representative's register.  Adjoints stay per slot, so each
    // slot keeps its own adjoint rule and the reverse sweep is unchanged.
    std::vector<uint32_t> rep;
    std::vector<uint8_t> vlive;      // representative whose value is needed
    std::vector<uint32_t> last_use;  // last forward reader of a value, or N for the loss

    explicit Info(const Tape &tape) : t(tape), N(uint32_t(tape.ops.size())), P(tape.n_params) {}

    // operand values of op k (as representatives)
    template <class F>
    void for_operands(uint32_t k, F f) const {
        for_operands_raw(k, [&](uint32_t s) { f(rep[s]); });
    }
    // operand slots of op k as written in the tape
    template <class F>
    void for_operands_raw(uint32_t k, F f) const {
        const TapeOp &o = t.ops[k];
        switch (o.code) {
        case tp::CONST: case tp::PARAM: case tp::OBS:
            return;
        case tp::PACK:
            for (uint32_t i = 0; i < o.b; ++i) f(t.aux[o.a + i]);
            return;
        case tp::SELECT:
            f(o.a); f(o.b); f(o.c); f(o.d);
            return;
        case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: case tp::POW: case tp::DOT:
        case tp::MATMUL: case tp::OUTER:
            f(o.a); f(o.b);
            return;
        default:
            f(o.a);
        }
    }
    // operands that receive an adjoint contribution from op k
    template <class F>
    void for_targets(uint32_t k, F f) const {
        const TapeOp &o = t.ops[k];
        switch (o.code) {
        case tp::CONST: case tp::PARAM: case tp::OBS:
            return;
        case tp::PACK:
            for (uint32_t i = 0; i < o.b; ++i) f(t.aux[o.a + i]);
            return;
        case tp::SELECT:
            f(o.c); f(o.d);
            return;
        case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: case tp::POW: case tp::DOT:
        case tp::MATMUL: case tp::OUTER:
            f(o.a); f(o.b);
            return;
        default:
            f(o.a);
        }
    }
    // values the adjoint rule of op k reads (k itself = its output z), as
    // representatives
    template <class F>
    void for_revreads(uint32_t k, F f) const {
        for_revreads_raw(k, [&](uint32_t s) { f(rep[s]); });
    }
    template <class F>
    void for_revreads_raw(uint32_t k, F f) const {
        const TapeOp &o = t.ops[k];
        switch (o.code) {
        case tp::MUL: case tp::DOT: case tp::MATMUL: case tp::OUTER: case tp::SELECT:
            f(o.a); f(o.b);
            return;
        case tp::DIV: f(o.b); f(k); return;
        case tp::EXP: f(k); return;
        case tp::LOG: case tp::SIN: case tp::COS: case tp::ABS: case tp::LOGDET: f(o.a); return;
        case tp::SQRT: f(o.a); f(k); return;
        case tp::POW: f(o.a); f(o.b); f(k); return;
        case tp::INV: f(k); return;
        case tp::DET: f(o.a); f(k); return;
        default: return;
        }
    }

    void number_values() {
        rep.assign(N, 0);
        std::map<std::vector<uint32_t>, uint32_t> first;
        std::vector<uint32_t> key;
        for (uint32_t k = 0; k < N; ++k) {
            const TapeOp &o = t.ops[k];
            key.assign({o.code, o.rows, o.cols, o.imm});
            for_operands_raw(k, [&](uint32_t s) { key.push_back(rep[s]); });
            auto it = first.emplace(key, k).first;
            rep[k] = it->second;
        }
    }

    void analyse() {
        kind.assign(N, K_COMP);
        nel.assign(N, 1);
        for (uint32_t k = 0; k < N; ++k) {
            uint16_t c = t.ops[k].code;
            kind[k] = c == tp::CONST ? K_CONST : c == tp::OBS ? K_OBS : c == tp::PARAM ? K_PARAM : K_COMP;
            nel[k] = uint8_t(t.nel(k));
        }
        number_values();
        // structure of the trace: slots the loss depends on (every one keeps
        // its adjoint rule, duplicates included)
        live.assign(N, 0);
        live[t.loss] = 1;
        for (uint32_t k = N; k-- > 0;)
            if (live[k]) for_operands_raw(k, [&](uint32_t s) { live[s] = 1; });
        active.assign(N, 0);
        for (uint32_t k = 0; k < N; ++k) {
            if (kind[k] == K_PARAM) { active[k] = 1; continue; }
            if (kind[k] != K_COMP) continue;
            bool a = false;
            for_targets(k, [&](uint32_t s) { a = a || active[s]; });
            active[k] = a;
        }
        has_adj.assign(N, 0);
        need_rev.assign(N, 0);
        has_adj[t.loss] = active[t.loss];
        for (uint32_t k = N; k-- > 0;) {
            if (!live[k] || kind[k] != K_COMP || !has_adj[k] || !active[k]) continue;
            need_rev[k] = 1;
            for_targets(k, [&](uint32_t s) {
                if (active[s]) has_adj[s] = 1;
            });
        }
        // values to compute: the loss, what the adjoint rules read, and what
        // those depend on
        vlive.assign(N, 0);
        vlive[rep[t.loss]] = 1;
        for (uint32_t k = N; k-- > 0;) {
            if (need_rev[k]) for_revreads(k, [&](uint32_t s) { vlive[s] = 1; });
            if (vlive[k] && rep[k] == k) for_operands(k, [&](uint32_t s) { vlive[s] = 1; });
        }
        last_use.assign(N, 0);
        for (uint32_t k = 0; k < N; ++k)
            if (vlive[k] && rep[k] == k) for_operands(k, [&](uint32_t s) { last_use[s] = k; });
        last_use[rep[t.loss]] = N;
    }
};

// ------------------------------------------------------------------ allocation
struct Interval {
    uint32_t start, end, nel;
    uint32_t reg;
};

// First-fit placement of intervals (sorted by start) into contiguous blocks.
// Returns the register high-water mark; a register whose interval ends at t
// is reusable from t + 1 on.
uint32_t allocate(std::vector<Interval> &iv) {
    std::vector<uint32_t> order(iv.size());
    for (uint32_t i = 0; i < iv.size(); ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(),
                     [&](uint32_t x, uint32_t y) { return iv[x].start < iv[y].start; });
    std::vector<uint32_t> busy;  // first time the register is free again
    uint32_t hwm = 0;
    for (uint32_t id : order) {
        Interval &v = iv[id];
        uint32_t r = 0, run = 0, base = 0;
        for (r = 0; r < busy.size(); ++r) {
            if (busy[r] <= v.start) {
                if (run == 0) base = r;
                if (++run == v.nel) break;
            } else {
                run = 0;
            }
        }
        if (run < v.nel) {
            if (run == 0) base = uint32_t(busy.size());
            busy.resize(base + v.nel, 0);
        }
        for (uint32_t i = 0; i < v.nel; ++i) busy[base + i] = v.end + 1;
        v.reg = base;
        hwm = std::max(hwm, base + v.nel);
    }
    return hwm;
}

// elementwise ops and the select have scalar fast-path opcodes
bool scalar_fast(uint16_t c) {
    switch (c) {
    case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: case tp::NEG: case tp::EXP: case tp::LOG:
    case tp::SQRT: case tp::SIN: case tp::COS: case tp::ABS: case tp::SELECT:
        return true;
    }
    return false;
}
bool binary_code(uint16_t c) { return c == tp::ADD || c == tp::SUB || c == tp::MUL || c == tp::DIV; }

uint32_t fwd_opcode(uint16_t c) {
    switch (c) {
    case tp::ADD: return isa::F_ADD;
    case tp::SUB: return isa::F_SUB;
    case tp::MUL: return isa::F_MUL;
    case tp::DIV: return isa::F_DIV;
    case tp::NEG: return isa::F_NEG;
    case tp::EXP: return isa::F_EXP;
    case tp::LOG: return isa::F_LOG;
    case tp::SQRT: return isa::F_SQRT;
    case tp::SIN: return isa::F_SIN;
    case tp::COS: return isa::F_COS;
    case tp::ABS: return isa::F_ABS;
    case tp::POW: return isa::F_POW;
    case tp::DOT: return isa::F_DOT;
    case tp::MATMUL: return isa::F_MATMUL;
    case tp::TRANSPOSE: return isa::F_TRANSPOSE;
    case tp::TRACE: return isa::F_TRACE;
    case tp::INV: return isa::F_INV;
    case tp::DET: return isa::F_DET;
    case tp::LOGDET: return isa::F_LOGDET;
    case tp::OUTER: return isa::F_OUTER;
    case tp::PACK: return isa::F_PACK;
    case tp::INDEX: return isa::F_INDEX;
    case tp::SELECT: return isa::F_SELECT;
    }
    return isa::END;
}

// ------------------------------------------------------------------ builder
// Abstract instruction before register assignment.
enum RIKind : uint8_t { I_LDP, I_LDC, I_CKST, I_FWD, I_STLOSS, I_ZEROP, I_SEED, I_CKLD, I_REV, I_STG };
struct AI {
    uint8_t kind;
    uint32_t k;   // slot / param index
    uint32_t j;   // segment (reverse phase) or checkpoint row
    uint8_t nb = 0;          // further ops bundled with k (I_FWD, I_REV)
    bool seq = false;        // reverse bundle whose rules' targets may repeat
    uint32_t kb[3] = {0, 0, 0};
    // the ops of a forward or reverse instruction
    uint32_t nops() const { return 1u + nb; }
    uint32_t op(uint32_t i) const { return i == 0 ? k : kb[i - 1]; }
};

struct Builder {
    const Info &I;
    const Tape &t;
    uint32_t N, P;
    // plan
    std::vector<uint32_t> cuts;       // segment starts, cuts[0] = 0
    std::vector<uint32_t> seg_of;
    std::vector<uint8_t> resident;
    std::vector<std::vector<uint32_t>> livein, recomp, revops;
    std::vector<uint32_t> res_off;    // resident slot -> offset in resident block
    uint32_t res_elems = 0;

    explicit Builder(const Info &info) : I(info), t(info.t), N(info.N), P(info.P) {}

    // a computed value the program needs (representatives only)
    bool comp_live(uint32_t s) const { return I.kind[s] == K_COMP && I.vlive[s]; }

    void set_cuts(const std::vector<uint32_t> &c) {
        cuts = c;
        seg_of.assign(N, 0);
        uint32_t j = 0;
        for (uint32_t k = 0; k < N; ++k) {
            while (j + 1 < cuts.size() && cuts[j + 1] <= k) ++j;
            seg_of[k] = j;
        }
    }

    void plan(bool with_residents) {
        uint32_t m = uint32_t(cuts.size());
        if (!with_residents) resident.assign(N, 0);
        livein.assign(m, {});
        recomp.assign(m, {});
        revops.assign(m, {});
        std::vector<uint32_t> mark(N, UINT32_MAX), inmark(N, UINT32_MAX), stack;
        for (uint32_t j = 0; j < m; ++j) {
            uint32_t lo = cuts[j], hi = j + 1 < m ? cuts[j + 1] : N;
            auto need = [&](uint32_t s) {
                if (I.kind[s] == K_OBS) {   // observations are reloaded, never checkpointed
                    if (mark[s] != j) { mark[s] = j; stack.push_back(s); }
                    return;
                }
                if (I.kind[s] != K_COMP || resident[s]) return;
                if (s >= lo) {
                    if (mark[s] != j) { mark[s] = j; stack.push_back(s); }
                } else if (inmark[s] != j) {
                    inmark[s] = j;
                    livein[j].push_back(s);
                }
            };
            for (uint32_t k = hi; k-- > lo;)
                if (I.need_rev[k]) {
                    revops[j].push_back(k);
                    I.for_revreads(k, need);
                }
            while (!stack.empty()) {
                uint32_t s = stack.back();
                stack.pop_back();
                recomp[j].push_back(s);
                I.for_operands(s, need);
            }
            std::sort(recomp[j].begin(), recomp[j].end());
            std::sort(livein[j].begin(), livein[j].end());
        }
    }

    void choose_residents(uint32_t K) {
        std::vector<uint32_t> cnt(N, 0);
        for (auto &v : livein)
            for (uint32_t s : v) cnt[s]++;
        resident.assign(N, 0);
        res_off.assign(N, 0);
        res_elems = 0;
        for (uint32_t s = 0; s < N; ++s)
            if (cnt[s] > K) {
                resident[s] = 1;
                res_off[s] = res_elems;
                res_elems += I.nel[s];
            }
    }

    std::vector<uint32_t> choose_cuts(uint64_t S) const {
        std::vector<int64_t> diff(N + 2, 0);
        for (uint32_t s = 0; s < N; ++s) {
            if (!comp_live(s) || resident[s]) continue;
            uint32_t lu = std::min(I.last_use[s], N);
            if (lu > s) {
                diff[s + 1] += I.nel[s];
                diff[lu + 1] -= I.nel[s];
            }
        }
        std::vector<int64_t> w(N + 1, 0);
        int64_t run = 0;
        for (uint32_t p = 0; p <= N; ++p) {
            run += diff[p];
            w[p] = run;
        }
        std::vector<uint32_t> c{0};
        uint64_t acc = 0;
        int64_t best = -1;
        uint32_t start = 0;
        for (uint32_t k = 0; k < N; ++k) {
            if (comp_live(k)) acc += I.nel[k];
            uint32_t p = k + 1;
            if (p >= N) break;
            if (acc * 2 >= S && p > start) {
                if (best < 0 || w[p] <= w[best]) best = p;
            }
            if (acc >= S && best > 0) {
                c.push_back(uint32_t(best));
                start = uint32_t(best);
                acc = 0;
                for (uint32_t q = start; q <= k; ++q)
                    if (comp_live(q)) acc += I.nel[q];
                best = -1;
            }
        }
        return c;
    }
};

// Bundle class of an op in the forward program: 1 fused multiply-add form of
// a scalar op (add, sub, mul, neg), 2 scalar division, 3 observation load,
// 0 none.
int fwd_class(const Info &I, uint32_t k) {
    const TapeOp &o = I.t.ops[k];
    if (I.kind[k] == K_OBS) return 3;
    if (I.kind[k] != K_COMP || I.nel[k] != 1 || I.nel[o.a] != 1) return 0;
    switch (o.code) {
    case tp::ADD: case tp::SUB: case tp::MUL: case tp::NEG: return 1;
    case tp::DIV: return 2;
    }
    return 0;
}
// Bundle class of a scalar op's adjoint rule: 1 linear (add, sub, mul, neg,
// exp), 2 division, 0 none.
int rev_class(const Info &I, uint32_t k) {
    const TapeOp &o = I.t.ops[k];
    if (I.kind[k] != K_COMP || I.nel[k] != 1 || I.nel[o.a] != 1) return 0;
    switch (o.code) {
    case tp::ADD: case tp::SUB: case tp::MUL: case tp::NEG: case tp::EXP: return 1;
    case tp::DIV: return 2;
    }
    return 0;
}
constexpr uint32_t kBundleMax = 3;
constexpr uint32_t kObsBundleMax = 4;
constexpr uint32_t kBundleWindow = 24;

// Reorder each run of forward instructions (list scheduling, earliest ready
// op first, data dependences kept) and bundle up to kBundleMax independent
// scalar ops of one class into one instruction.  Every op still computes
// exactly what it computed before, so results are unchanged bit for bit.
std::vector<AI> bundle_forward(const Info &I, const std::vector<AI> &in) {
    std::vector<AI> out;
    out.reserve(in.size());
    size_t i = 0;
    std::vector<uint32_t> pos_of(I.N, UINT32_MAX);
    while (i < in.size()) {
        if (in[i].kind != I_FWD) {
            out.push_back(in[i++]);
            continue;
        }
        size_t e = i;
        while (e < in.size() && in[e].kind == I_FWD && in[e].j == in[i].j) ++e;
        const uint32_t n = uint32_t(e - i);
        for (uint32_t q = 0; q < n; ++q) pos_of[in[i + q].k] = q;
        std::vector<uint8_t> done(n, 0);
        std::vector<uint32_t> pending(n, 0);   // operands still to be emitted
        std::vector<uint32_t> ucnt(n + 1, 0), users;
        for (uint32_t q = 0; q < n; ++q)
            I.for_operands(in[i + q].k, [&](uint32_t s) {
                if (pos_of[s] != UINT32_MAX) {
                    pending[q]++;
                    ucnt[pos_of[s] + 1]++;
                }
            });
        for (uint32_t q = 0; q < n; ++q) ucnt[q + 1] += ucnt[q];
        users.resize(ucnt[n]);
        {
            std::vector<uint32_t> fill(ucnt.begin(), ucnt.end() - 1);
            for (uint32_t q = 0; q < n; ++q)
                I.for_operands(in[i + q].k, [&](uint32_t s) {
                    if (pos_of[s] != UINT32_MAX) users[fill[pos_of[s]]++] = q;
                });
        }
        auto retire = [&](uint32_t q) {
            done[q] = 1;
            for (uint32_t u = ucnt[q]; u < ucnt[q + 1]; ++u) pending[users[u]]--;
        };
        uint32_t first = 0;
        for (uint32_t emitted = 0; emitted < n;) {
            while (done[first]) ++first;
            uint32_t x = first;
            while (pending[x] != 0) ++x;         // earliest ready op
            // a ready observation load in the window goes first: it is cheap
            // and makes its users ready to be bundled
            for (uint32_t r = x; r < n && r < x + kBundleWindow; ++r)
                if (!done[r] && pending[r] == 0 && I.kind[in[i + r].k] == K_OBS) {
                    x = r;
                    break;
                }
            AI a = in[i + x];
            const int cls = fwd_class(I, a.k);
            const uint32_t cap = cls == 3 ? kObsBundleMax : kBundleMax;
            if (cls)
                for (uint32_t r = x + 1; r < n && r < x + kBundleWindow && a.nb + 1u < cap; ++r)
                    if (!done[r] && pending[r] == 0 && fwd_class(I, in[i + r].k) == cls) {
                        a.kb[a.nb++] = in[i + r].k;
                        done[r] = 2;             // taken; retired with the bundle
                    }
            retire(x);
            for (uint32_t r = x + 1; r < n && r < x + kBundleWindow; ++r)
                if (done[r] == 2) retire(r);
            out.push_back(a);
            emitted += a.nops();
        }
        for (uint32_t q = 0; q < n; ++q) pos_of[in[i + q].k] = UINT32_MAX;
        i = e;
    }
    return out;
}

// Bundle scalar adjoint rules of each run of reverse instructions.  An op may
// be hoisted next to an earlier one only when its own adjoint is complete
// (every op contributing to it has been emitted) and no op it jumps over
// touches any of its targets; so every adjoint still receives its
// contributions in the same order and the results are unchanged bit for
// bit.  Within a bundle the rules are applied in their original order; a
// bundle whose targets repeat (x * x, or two rules feeding one adjoint) is
// marked sequential, the others let the handler read every target first.
std::vector<AI> bundle_reverse(const Info &I, const std::vector<AI> &in) {
    std::vector<AI> out;
    out.reserve(in.size());
    auto tid = [&](uint32_t s) -> int64_t {   // adjoint identity of a target, -1 if none
        if (I.kind[s] == K_PARAM) return int64_t(I.N) + I.t.ops[s].imm;
        if (I.kind[s] == K_COMP && I.active[s]) return s;
        return -1;
    };
    size_t i = 0;
    while (i < in.size()) {
        if (in[i].kind != I_REV) {
            out.push_back(in[i++]);
            continue;
        }
        size_t e = i;
        while (e < in.size() && in[e].kind == I_REV && in[e].j == in[i].j) ++e;
        const uint32_t n = uint32_t(e - i);
        std::vector<std::vector<int64_t>> T(n);
        std::vector<uint8_t> self_clash(n, 0);
        std::unordered_map<int64_t, std::vector<uint32_t>> by_target;
        for (uint32_t q = 0; q < n; ++q) {
            I.for_targets(in[i + q].k, [&](uint32_t s) {
                int64_t id = tid(s);
                if (id < 0) return;
                for (int64_t x : T[q]) self_clash[q] = self_clash[q] || x == id;
                T[q].push_back(id);
            });
            for (int64_t id : T[q]) by_target[id].push_back(q);
        }
        std::vector<uint32_t> pend(n, 0);
        for (uint32_t q = 0; q < n; ++q) {
            auto it = by_target.find(int64_t(in[i + q].k));
            if (it != by_target.end())
                for (uint32_t p : it->second)
                    if (p < q) pend[q]++;
        }
        std::vector<uint8_t> done(n, 0);
        auto retire = [&](uint32_t q) {
            done[q] = 1;
            for (int64_t id : T[q]) {
                if (id >= int64_t(I.N)) continue;
                // ops in this run whose output is `id` lose one pending contributor
                for (uint32_t r = q + 1; r < n && r < q + 4 * kBundleWindow; ++r)
                    if (int64_t(in[i + r].k) == id && pend[r] > 0) pend[r]--;
            }
        };
        auto clashes = [&](uint32_t r, const std::vector<int64_t> &ids) {
            for (int64_t id : T[r])
                for (int64_t x : ids)
                    if (id == x) return true;
            return false;
        };
        uint32_t first = 0;
        std::vector<int64_t> skipped, taken;
        for (uint32_t emitted = 0; emitted < n;) {
            while (done[first]) ++first;
            const uint32_t x = first;
            AI a = in[i + x];
            const int cls = rev_class(I, a.k);
            uint32_t picked[kBundleMax - 1];
            a.seq = self_clash[x];
            if (cls) {
                skipped.clear();
                taken.assign(T[x].begin(), T[x].end());
                for (uint32_t r = x + 1; r < n && r < x + kBundleWindow && a.nb + 1 < kBundleMax; ++r) {
                    if (done[r]) continue;
                    if (pend[r] == 0 && rev_class(I, in[i + r].k) == cls && !clashes(r, skipped)) {
                        a.seq = a.seq || self_clash[r] || clashes(r, taken);
                        picked[a.nb] = r;
                        a.kb[a.nb++] = in[i + r].k;
                        taken.insert(taken.end(), T[r].begin(), T[r].end());
                        continue;
                    }
                    skipped.insert(skipped.end(), T[r].begin(), T[r].end());
                    skipped.push_back(int64_t(in[i + r].k));
                }
            }
            out.push_back(a);
            retire(x);
            for (uint32_t b = 0; b < a.nb; ++b) retire(picked[b]);
            emitted += a.nops();
        }
        i = e;
    }
    return out;
}

struct Emitter {
    std::vector<uint32_t> code, aux;
    void put(uint32_t a, uint32_t b = 0, uint32_t c = 0, uint32_t d = 0, uint32_t e = 0, uint32_t f = 0,
             uint32_t g = 0, uint32_t h = 0) {
        uint32_t w[8] = {a, b, c, d, e, f, g, h};
        code.insert(code.end(), w, w + 8);
    }
};

// Terminate the program: NOPs up to the next fetch chunk, a chunk of END,
// and the chunk the fetch reads ahead (also END).
bool repeatable(uint32_t op) {
    return (op >= isa::FB1 && op <= isa::RDBS3) || (op >= isa::OB2 && op <= isa::OB4) || op == isa::F_MATMUL ||
           op == isa::R_MATMUL;
}

void finish(Emitter &E, Schedule &S) {
    const size_t n = E.code.size() / isa::kWords;
    for (size_t k = 0; k + 1 < n; ++k) {
        uint32_t &w0 = E.code[k * isa::kWords];
        const uint32_t op = w0 & 0xFF;
        if (repeatable(op) && (k + 1) % isa::kChunkInstr != 0 && (E.code[(k + 1) * isa::kWords] & 0xFF) == op)
            w0 |= isa::kRepeat;
    }
    while (E.code.size() % isa::kChunkWords) E.put(isa::w0(isa::NOP, 0, 0));
    S.n_instr = E.code.size() / isa::kWords + 1;   // through the END
    for (uint32_t i = 0; i < 2 * isa::kChunkInstr; ++i) E.put(isa::w0(isa::END, 0, 0));
    S.code = std::move(E.code);
    S.aux = std::move(E.aux);
}

// Build the forward phase (shared by both programs) and, for the gradient
// program, the reverse phase; returns the schedule with registers assigned.
Schedule build(const Info &I, Builder &B, bool with_grad) {
    const Tape &t = I.t;
    const uint32_t N = I.N, P = I.P;
    // static registers: param values, param adjoints, a sink for adjoint
    // contributions nobody needs, the constant pool, residents
    // the pool holds the tape's constants, then 1, -1 and -0 for bundles
    const uint32_t nt = uint32_t(t.consts.size()), nc = nt + 3;
    const uint32_t kSink = 2 * P, kConst0 = 2 * P + 1;
    const uint32_t kOne = kConst0 + nt, kMinusOne = kOne + 1, kNegZero = kOne + 2;
    const uint32_t kStatic = 2 * P + 1 + nc + B.res_elems;
    const uint32_t m = uint32_t(B.cuts.size());
    Schedule S;
    S.n_segments = with_grad ? m : 1;
    S.static_regs = kStatic;
    S.consts = t.consts;
    S.consts.push_back(1.0);
    S.consts.push_back(-1.0);
    S.consts.push_back(-0.0);

    // ---- forward phase: abstract instructions + value intervals
    std::vector<AI> fa;
    std::vector<uint32_t> ckrow_of;   // per (segment, livein index) row, flattened
    std::vector<uint32_t> ckrow_base(m + 1, 0);
    if (with_grad) {
        uint32_t row = 0;
        for (uint32_t j = 0; j < m; ++j) {
            ckrow_base[j] = row;
            for (uint32_t s : B.livein[j]) row += I.nel[s];
        }
        ckrow_base[m] = row;
        S.n_ckpt_rows = row;
    }
    for (uint32_t p = 0; p < P; ++p) fa.push_back({I_LDP, p, 0});
    for (uint32_t i = 0; i < nc; i += 255) fa.push_back({I_LDC, i, std::min<uint32_t>(255, nc - i)});
    uint32_t next_cut = 1;
    for (uint32_t k = 0; k < N; ++k) {
        if (with_grad) {
            while (next_cut < m && B.cuts[next_cut] == k) {
                for (uint32_t i = 0; i < B.livein[next_cut].size(); ++i) fa.push_back({I_CKST, next_cut, i});
                ++next_cut;
            }
        }
        if (B.comp_live(k) || (I.kind[k] == K_OBS && I.vlive[k])) fa.push_back({I_FWD, k, 0});
    }
    fa.push_back({I_STLOSS, t.loss, 0});
    fa = bundle_forward(I, fa);
    // intervals for forward values
    std::vector<Interval> fiv;
    std::vector<int32_t> fiv_of(N, -1);
    for (uint32_t ti = 0; ti < fa.size(); ++ti) {
        const AI &a = fa[ti];
        auto use = [&](uint32_t s) {
            if (fiv_of[s] >= 0) fiv[fiv_of[s]].end = std::max(fiv[fiv_of[s]].end, ti);
        };
        if (a.kind == I_FWD) {
            for (uint32_t b = 0; b < a.nops(); ++b) I.for_operands(a.op(b), use);
            for (uint32_t b = 0; b < a.nops(); ++b) {
                const uint32_t k = a.op(b);
                if (fiv_of[k] >= 0 || (with_grad && B.resident[k])) continue;
                fiv_of[k] = int32_t(fiv.size());
                fiv.push_back({ti, ti, I.nel[k], 0});
            }
        } else if (a.kind == I_CKST) {
            use(B.livein[a.k][a.j]);
        } else if (a.kind == I_STLOSS) {
            use(a.k);
        }
    }
    uint32_t fhwm = allocate(fiv);
    S.fwd_regs = fhwm;

    auto res_reg = [&](uint32_t s) { return kConst0 + nc + B.res_off[s]; };
    auto fwd_operand = [&](uint32_t s) -> uint32_t {
        s = I.rep[s];
        switch (I.kind[s]) {
        case K_CONST: return kConst0 + t.ops[s].imm;
        case K_PARAM: return t.ops[s].imm;
        default:
            if (with_grad && B.resident[s]) return res_reg(s);
            return kStatic + fiv[fiv_of[s]].reg;
        }
    };

    Emitter E;
    auto emit_fwd = [&](uint32_t k, auto operand, uint32_t dst) {
        const TapeOp &o = t.ops[k];
        uint32_t op = fwd_opcode(o.code), n = I.nel[k];
        if (o.code == tp::OBS) {
            E.put(isa::w0(isa::LDOBS, 0, 1), dst, 0, 0, 0, 0, 0, o.imm);
            return;
        }
        if (n == 1 && scalar_fast(o.code) && (o.code == tp::SELECT || I.nel[o.a] == 1)) {
            uint32_t sop = op == isa::F_SELECT ? uint32_t(isa::S_SELECT) : op - isa::F_ADD + isa::S_ADD;
            if (o.code == tp::SELECT)
                E.put(isa::w0(sop, 0, 1), dst, operand(o.a), operand(o.b), operand(o.c), operand(o.d));
            else
                E.put(isa::w0(sop, 0, 1), dst, operand(o.a), binary_code(o.code) ? operand(o.b) : 0);
            return;
        }
        switch (o.code) {
        case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: {
            uint32_t mode = isa::MODE_SAME;
            if (I.nel[o.a] != I.nel[o.b] || t.ops[o.a].rows != t.ops[o.b].rows)
                mode = I.nel[o.a] == 1 ? isa::MODE_A_SCALAR : isa::MODE_B_SCALAR;
            E.put(isa::w0(op, mode, n), dst, operand(o.a), operand(o.b));
            break;
        }
        case tp::POW:
            E.put(isa::w0(op, 0, 1), dst, operand(o.a), operand(o.b));
            break;
        case tp::DOT:
            E.put(isa::w0(op, 0, I.nel[o.a]), dst, operand(o.a), operand(o.b));
            break;
        case tp::MATMUL:
            E.put(isa::w0(op, 0, n), dst, operand(o.a), operand(o.b), 0, 0, 0,
                  isa::dims(t.ops[o.a].rows, t.ops[o.a].cols, t.ops[o.b].cols));
            break;
        case tp::TRANSPOSE: case tp::OUTER:
            E.put(isa::w0(op, 0, n), dst, operand(o.a), o.code == tp::OUTER ? operand(o.b) : 0, 0, 0, 0,
                  isa::dims(t.ops[o.a].rows, o.code == tp::OUTER ? t.ops[o.b].rows : t.ops[o.a].cols, 0));
            break;
        case tp::TRACE: case tp::INV: case tp::DET: case tp::LOGDET:
            E.put(isa::w0(op, 0, n), dst, operand(o.a), 0, 0, 0, 0, t.ops[o.a].rows);
            break;
        case tp::PACK: {
            uint32_t off = uint32_t(E.aux.size());
            for (uint32_t i = 0; i < o.b; ++i) E.aux.push_back(operand(t.aux[o.a + i]));
            E.put(isa::w0(op, 0, n), dst, 0, 0, 0, 0, 0, off);
            break;
        }
        case tp::INDEX:
            E.put(isa::w0(op, 0, 1), dst, operand(o.a), 0, 0, 0, 0, o.imm);
            break;
        case tp::SELECT:
            E.put(isa::w0(op, 0, n), dst, operand(o.a), operand(o.b), operand(o.c), operand(o.d));
            break;
        default:  // elementwise unary
            E.put(isa::w0(op, 0, n), dst, operand(o.a));
        }
    };

    // a forward bundle: the fused multiply-add form of each op, or divisions;
    // single ops (and bundles naming registers beyond the 16-bit fields) use
    // the one-op instructions
    auto emit_bundle = [&](const AI &a, auto operand) {
        const uint32_t nb = a.nops();
        const int cls = nb > 1 ? fwd_class(I, a.k) : 0;
        if (cls == 3) {   // observation loads: fields (d, observation index)
            bool ok = true;
            uint32_t w[8] = {isa::OB2 + nb - 2, 0, 0, 0, 0, 0, 0, 0};
            for (uint32_t b = 0; b < nb; ++b) {
                const uint32_t d = operand(a.op(b)), idx = t.ops[a.op(b)].imm;
                ok = ok && d < isa::kFieldMaxReg && idx < isa::kFieldMaxReg;
                w[1 + b] = d | (idx << 16);
            }
            if (ok) {
                E.put(w[0], w[1], w[2], w[3], w[4], w[5], w[6], w[7]);
                S.n_bundles++;
                S.n_bundled_ops += nb;
                return;
            }
            for (uint32_t b = 0; b < nb; ++b) emit_fwd(a.op(b), operand, operand(a.op(b)));
            return;
        }
        uint32_t f[15] = {};
        uint32_t nf = 0;
        bool fits = cls != 0;
        for (uint32_t b = 0; b < nb && fits; ++b) {
            const uint32_t k = a.op(b);
            const TapeOp &o = t.ops[k];
            uint32_t x[4];
            if (cls == 2) {
                x[0] = operand(k); x[1] = operand(o.a); x[2] = operand(o.b);
            } else {
                switch (o.code) {
                case tp::ADD: x[1] = operand(o.a); x[2] = kOne; x[3] = operand(o.b); break;
                case tp::SUB: x[1] = operand(o.b); x[2] = kMinusOne; x[3] = operand(o.a); break;
                case tp::MUL: x[1] = operand(o.a); x[2] = operand(o.b); x[3] = kNegZero; break;
                default: x[1] = operand(o.a); x[2] = kMinusOne; x[3] = kNegZero; break;   // NEG
                }
                x[0] = operand(k);
            }
            for (uint32_t q = 0; q < (cls == 2 ? 3u : 4u); ++q) {
                fits = fits && x[q] < isa::kFieldMaxReg;
                f[nf++] = x[q];
            }
        }
        if (!fits) {
            for (uint32_t b = 0; b < nb; ++b) emit_fwd(a.op(b), operand, operand(a.op(b)));
            return;
        }
        const uint32_t op = (cls == 2 ? isa::DB1 : isa::FB1) + nb - 1;
        uint32_t w[8] = {op, 0, 0, 0, 0, 0, 0, 0};
        for (uint32_t q = 0; q < nf; ++q) w[1 + q / 2] |= f[q] << (16 * (q & 1));
        E.put(w[0], w[1], w[2], w[3], w[4], w[5], w[6], w[7]);
        S.n_bundles++;
        S.n_bundled_ops += nb;
    };
    for (const AI &a : fa) {
        switch (a.kind) {
        case I_LDP: E.put(isa::w0(isa::LDPARAM, 0, 1), a.k, 0, 0, 0, 0, 0, a.k); break;
        case I_LDC: E.put(isa::w0(isa::LDCONST, 0, a.j), kConst0 + a.k, 0, 0, 0, 0, 0, a.k); break;
        case I_CKST: {
            uint32_t s = B.livein[a.k][a.j];
            uint32_t row = ckrow_base[a.k];
            for (uint32_t i = 0; i < a.j; ++i) row += I.nel[B.livein[a.k][i]];
            E.put(isa::w0(isa::CKPT_ST, 0, I.nel[s]), 0, fwd_operand(s), 0, 0, 0, 0, row);
            S.ckpt_elems_stored += I.nel[s];
            break;
        }
        case I_FWD:
            emit_bundle(a, fwd_operand);
            S.n_fwd_ops += a.nops();
            break;
        case I_STLOSS: E.put(isa::w0(isa::ST_LOSS, 0, 1), 0, fwd_operand(a.k)); break;
        }
    }
    if (!with_grad) {
        S.n_regs = kStatic + fhwm;
        finish(E, S);
        return S;
    }

    // ---- reverse phase
    std::vector<AI> ra;
    ra.push_back({I_ZEROP, 0, 0});
    ra.push_back({I_SEED, t.loss, 0});
    for (uint32_t j = m; j-- > 0;) {
        for (uint32_t i = 0; i < B.livein[j].size(); ++i) ra.push_back({I_CKLD, j, i});
        for (uint32_t s : B.recomp[j]) ra.push_back({I_FWD, s, j});
        for (uint32_t k : B.revops[j]) ra.push_back({I_REV, k, j});
    }
    for (uint32_t p = 0; p < P; ++p) ra.push_back({I_STG, p, 0});
    ra = bundle_forward(I, ra);
    ra = bundle_reverse(I, ra);

    // value intervals keyed by (slot, segment); adjoint intervals keyed by slot
    std::vector<Interval> riv;
    std::unordered_map<uint64_t, uint32_t> val_of;
    std::vector<int32_t> adj_of(N, -1);
    auto key = [](uint32_t s, uint32_t j) { return (uint64_t(s) << 32) | j; };
    auto vuse = [&](uint32_t s, uint32_t j, uint32_t ti) {
        if ((I.kind[s] != K_COMP && I.kind[s] != K_OBS) || B.resident[s]) return;
        auto it = val_of.find(key(s, j));
        riv[it->second].end = std::max(riv[it->second].end, ti);
    };
    // first contribution flags: (instruction index, target position) -> init
    std::vector<uint8_t> touched(N, 0);
    auto contrib = [&](uint32_t s, uint32_t ti) {
        if (I.kind[s] != K_COMP || !I.active[s]) return;
        if (!touched[s]) {
            touched[s] = 1;
            adj_of[s] = int32_t(riv.size());
            riv.push_back({ti, ti, I.nel[s], 0});
        }
    };
    for (uint32_t ti = 0; ti < ra.size(); ++ti) {
        const AI &a = ra[ti];
        switch (a.kind) {
        case I_SEED:
            contrib(a.k, ti);
            break;
        case I_CKLD: {
            uint32_t s = B.livein[a.k][a.j];
            val_of[key(s, a.k)] = uint32_t(riv.size());
            riv.push_back({ti, ti, I.nel[s], 0});
            break;
        }
        case I_FWD:
            for (uint32_t b = 0; b < a.nops(); ++b)
                I.for_operands(a.op(b), [&](uint32_t s) { vuse(s, a.j, ti); });
            for (uint32_t b = 0; b < a.nops(); ++b) {
                val_of[key(a.op(b), a.j)] = uint32_t(riv.size());
                riv.push_back({ti, ti, I.nel[a.op(b)], 0});
            }
            break;
        case I_REV: {
            for (uint32_t b = 0; b < a.nops(); ++b) {
                const uint32_t k = a.op(b);
                I.for_revreads(k, [&](uint32_t s) { vuse(s, a.j, ti); });
                I.for_targets(k, [&](uint32_t s) { contrib(s, ti); });
                int32_t g = adj_of[k];
                riv[g].end = std::max(riv[g].end, ti);
            }
            break;
        }
        default:
            break;
        }
    }
    uint32_t rhwm = allocate(riv);
    S.rev_regs = rhwm;
    S.n_regs = kStatic + std::max(fhwm, rhwm);

    auto rev_operand = [&](uint32_t s, uint32_t j) -> uint32_t {
        s = I.rep[s];
        switch (I.kind[s]) {
        case K_CONST: return kConst0 + t.ops[s].imm;
        case K_PARAM: return t.ops[s].imm;
        default:
            if (B.resident[s]) return res_reg(s);
            return kStatic + riv[val_of.at(key(s, j))].reg;
        }
    };
    std::fill(touched.begin(), touched.end(), 0);
    auto target_word = [&](uint32_t s) -> uint32_t {
        if (I.kind[s] == K_PARAM) return P + t.ops[s].imm;
        if (I.kind[s] != K_COMP || !I.active[s]) return isa::kNone;
        uint32_t r = kStatic + riv[adj_of[s]].reg;
        if (!touched[s]) {
            touched[s] = 1;
            return r | isa::kInit;
        }
        return r;
    };
    auto target = target_word;
    auto adjreg = [&](uint32_t s) { return kStatic + riv[adj_of[s]].reg; };

    // one op's adjoint rule as a single instruction
    auto emit_rev1 = [&](uint32_t k, uint32_t j) {
        do {
            const TapeOp &o = t.ops[k];
            const uint32_t n = I.nel[k];
            uint32_t g = adjreg(k);
            auto v = [&](uint32_t s) { return rev_operand(s, j); };
            uint32_t op = fwd_opcode(o.code) - isa::F_ADD + isa::R_ADD;
            S.n_rev_ops++;
            if (n == 1 && scalar_fast(o.code) && (o.code == tp::SELECT || I.nel[o.a] == 1)) {
                uint32_t sop = o.code == tp::SELECT ? uint32_t(isa::SR_SELECT)
                                                    : fwd_opcode(o.code) - isa::F_ADD + isa::SR_ADD;
                uint32_t va = 0, vb = 0, vz = 0, ta = isa::kNone, tb = isa::kNone;
                auto target = [&](uint32_t s) {
                    uint32_t x = target_word(s);
                    return x == isa::kNone ? kSink : x;
                };
                switch (o.code) {
                case tp::ADD: case tp::SUB: ta = target(o.a); tb = target(o.b); break;
                case tp::MUL: va = v(o.a); vb = v(o.b); ta = target(o.a); tb = target(o.b); break;
                case tp::DIV: vb = v(o.b); vz = v(k); ta = target(o.a); tb = target(o.b); break;
                case tp::NEG: ta = target(o.a); break;
                case tp::EXP: vz = v(k); ta = target(o.a); break;
                case tp::SQRT: va = v(o.a); vz = v(k); ta = target(o.a); break;
                case tp::SELECT: va = v(o.a); vb = v(o.b); ta = target(o.c); tb = target(o.d); break;
                default: va = v(o.a); ta = target(o.a); break;   // LOG SIN COS ABS
                }
                E.put(isa::w0(sop, 0, 1), g, va, vb, vz, ta, tb);
                break;
            }
            switch (o.code) {
            case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: {
                uint32_t mode = isa::MODE_SAME;
                if (I.nel[o.a] != I.nel[o.b] || t.ops[o.a].rows != t.ops[o.b].rows)
                    mode = I.nel[o.a] == 1 ? isa::MODE_A_SCALAR : isa::MODE_B_SCALAR;
                uint32_t va = (o.code == tp::MUL) ? v(o.a) : 0;
                uint32_t vb = (o.code == tp::MUL || o.code == tp::DIV) ? v(o.b) : 0;
                uint32_t vz = o.code == tp::DIV ? v(k) : 0;
                uint32_t ta = target(o.a), tb = target(o.b);
                E.put(isa::w0(op, mode, n), g, va, vb, vz, ta, tb);
                break;
            }
            case tp::POW: {
                uint32_t va = v(o.a), vb = v(o.b), vz = v(k);
                uint32_t ta = target(o.a), tb = target(o.b);
                E.put(isa::w0(op, 0, 1), g, va, vb, vz, ta, tb);
                break;
            }
            case tp::DOT: {
                uint32_t va = v(o.a), vb = v(o.b);
                uint32_t ta = target(o.a), tb = target(o.b);
                E.put(isa::w0(op, 0, I.nel[o.a]), g, va, vb, 0, ta, tb);
                break;
            }
            case tp::MATMUL: {
                uint32_t va = v(o.a), vb = v(o.b);
                uint32_t ta = target(o.a), tb = target(o.b);
                E.put(isa::w0(op, 0, n), g, va, vb, 0, ta, tb,
                      isa::dims(t.ops[o.a].rows, t.ops[o.a].cols, t.ops[o.b].cols));
                break;
            }
            case tp::OUTER: {
                uint32_t va = v(o.a), vb = v(o.b);
                uint32_t ta = target(o.a), tb = target(o.b);
                E.put(isa::w0(op, 0, n), g, va, vb, 0, ta, tb, isa::dims(t.ops[o.a].rows, t.ops[o.b].rows, 0));
                break;
            }
            case tp::TRANSPOSE:
                E.put(isa::w0(op, 0, n), g, 0, 0, 0, target(o.a), 0,
                      isa::dims(t.ops[o.a].rows, t.ops[o.a].cols, 0));
                break;
            case tp::TRACE:
                E.put(isa::w0(op, 0, 1), g, 0, 0, 0, target(o.a), 0, t.ops[o.a].rows);
                break;
            case tp::INV:
                E.put(isa::w0(op, 0, n), g, 0, 0, v(k), target(o.a), 0, t.ops[o.a].rows);
                break;
            case tp::DET: {
                uint32_t va = v(o.a), vz = v(k);
                E.put(isa::w0(op, 0, 1), g, va, 0, vz, target(o.a), 0, t.ops[o.a].rows);
                break;
            }
            case tp::LOGDET:
                E.put(isa::w0(op, 0, 1), g, v(o.a), 0, 0, target(o.a), 0, t.ops[o.a].rows);
                break;
            case tp::PACK: {
                uint32_t off = uint32_t(E.aux.size());
                for (uint32_t i = 0; i < o.b; ++i) E.aux.push_back(target(t.aux[o.a + i]));
                E.put(isa::w0(op, 0, n), g, 0, 0, 0, 0, 0, off);
                break;
            }
            case tp::INDEX:
                E.put(isa::w0(op, 0, I.nel[o.a]), g, 0, 0, 0, target(o.a), 0, o.imm);
                break;
            case tp::SELECT: {
                uint32_t va = v(o.a), vb = v(o.b);
                uint32_t tc = target(o.c), td = target(o.d);
                E.put(isa::w0(op, 0, n), g, va, vb, 0, tc, td);
                break;
            }
            case tp::EXP: case tp::SQRT: {
                uint32_t va = o.code == tp::SQRT ? v(o.a) : 0, vz = v(k);
                E.put(isa::w0(op, 0, n), g, va, 0, vz, target(o.a));
                break;
            }
            default:  // NEG, LOG, SIN, COS, ABS
                E.put(isa::w0(op, 0, n), g, o.code == tp::NEG ? 0 : v(o.a), 0, 0, target(o.a));
            }
        } while (false);
    };
    // value (not adjoint-first) register of a target, without side effects
    auto target_reg = [&](uint32_t s) -> uint32_t {
        if (I.kind[s] == K_PARAM) return P + t.ops[s].imm;
        if (I.kind[s] != K_COMP || !I.active[s]) return kSink;
        return kStatic + riv[adj_of[s]].reg;
    };


    for (const AI &a : ra) {
        switch (a.kind) {
        case I_ZEROP:
            for (uint32_t p0 = 0; p0 < P; p0 += 16)
                E.put(isa::w0(isa::ZERO, 0, std::min<uint32_t>(16, P - p0)), P + p0);
            break;
        case I_SEED:
            if (I.kind[a.k] == K_PARAM || (I.kind[a.k] == K_COMP && I.active[a.k]))
                E.put(isa::w0(isa::SEED, 0, 1), 0, 0, 0, 0, target(a.k));
            break;
        case I_CKLD: {
            uint32_t s = B.livein[a.k][a.j];
            uint32_t row = ckrow_base[a.k];
            for (uint32_t i = 0; i < a.j; ++i) row += I.nel[B.livein[a.k][i]];
            E.put(isa::w0(isa::CKPT_LD, 0, I.nel[s]), rev_operand(s, a.k), 0, 0, 0, 0, 0, row);
            S.ckpt_elems_loaded += I.nel[s];
            break;
        }
        case I_FWD: {
            auto opnd = [&](uint32_t s) { return rev_operand(s, a.j); };
            emit_bundle(a, opnd);
            S.n_recompute_ops += a.nops();
            break;
        }
        case I_REV: {
            const uint32_t nb = a.nops();
            const int cls = nb > 1 || a.seq ? rev_class(I, a.k) : 0;
            // the registers a rule reads: g, ya, yb
            auto rule_regs = [&](uint32_t k, uint32_t (&r)[3]) {
                const TapeOp &o = t.ops[k];
                auto v = [&](uint32_t s) { return rev_operand(s, a.j); };
                r[0] = adjreg(k);
                r[1] = kOne;
                r[2] = kOne;
                if (cls == 2) {
                    r[1] = v(o.b);
                    r[2] = v(k);
                    return;
                }
                switch (o.code) {
                case tp::SUB: r[2] = kMinusOne; break;
                case tp::MUL: r[1] = v(o.b); r[2] = v(o.a); break;
                case tp::NEG: r[1] = kMinusOne; break;
                case tp::EXP: r[1] = v(k); break;
                default: break;   // ADD
                }
            };
            bool fits = cls != 0;
            for (uint32_t b = 0; b < nb && fits; ++b) {
                const uint32_t k = a.op(b);
                const TapeOp &o = t.ops[k];
                uint32_t r[3];
                rule_regs(k, r);
                fits = r[0] < isa::kFieldMaxReg && r[1] < isa::kFieldMaxReg && r[2] < isa::kFieldMaxReg &&
                       target_reg(o.a) < isa::kFieldMaxReg &&
                       (!binary_code(o.code) || target_reg(o.b) < isa::kFieldMaxReg);
            }
            if (!fits) {
                for (uint32_t b = 0; b < nb; ++b) emit_rev1(a.op(b), a.j);
                break;
            }
            const uint32_t op0 = a.seq ? (cls == 2 ? isa::RDBS1 : isa::LBS1) : (cls == 2 ? isa::RDB1 : isa::LB1);
            uint32_t w[8] = {op0 + nb - 1, 0, 0, 0, 0, 0, 0, 0};
            auto put_field = [&](uint32_t i, uint32_t f) {
                if (i == 14)
                    w[0] |= f << 16;
                else
                    w[1 + i / 2] |= f << (16 * (i & 1));
            };
            // target register; its first contribution sets flag bit `bit` of w0
            auto tfield = [&](uint32_t s, uint32_t bit) {
                const uint32_t x = target_word(s);
                if (x == isa::kNone) return kSink;
                if (x & isa::kInit) w[0] |= 1u << bit;
                return x & ~isa::kInit;
            };
            for (uint32_t b = 0; b < nb; ++b) {
                const uint32_t k = a.op(b);
                const TapeOp &o = t.ops[k];
                uint32_t r[3];
                rule_regs(k, r);
                put_field(5 * b, r[0]);
                put_field(5 * b + 1, r[1]);
                put_field(5 * b + 2, r[2]);
                put_field(5 * b + 3, tfield(o.a, 8 + 2 * b));
                put_field(5 * b + 4, binary_code(o.code) ? tfield(o.b, 9 + 2 * b) : kSink);
            }
            E.put(w[0], w[1], w[2], w[3], w[4], w[5], w[6], w[7]);
            S.n_rev_ops += nb;
            S.n_bundles++;
            S.n_bundled_ops += nb;
            break;
        }
        case I_STG:
            E.put(isa::w0(isa::ST_GRAD, 0, 1), 0, P + a.k, 0, 0, 0, 0, a.k);
            break;
        default:
            break;
        }
    }
    finish(E, S);
    return S;
}

}  // namespace

Schedule schedule_forward(const Tape &t) {
    Info I(t);
    I.analyse();
    Builder B(I);
    B.set_cuts({0});
    B.resident.assign(I.N, 0);
    B.res_off.assign(I.N, 0);
    return build(I, B, false);
}

Schedule schedule_grad(const Tape &t, uint32_t reg_budget) {
    Info I(t);
    I.analyse();
    uint64_t total = 0;
    for (uint32_t k = 0; k < I.N; ++k)
        if (I.kind[k] == K_COMP && I.vlive[k]) total += I.nel[k];
    const uint32_t kResidentAfter = 2;   // checkpointed in more segments -> keep resident
    auto trial = [&](uint64_t S) {
        Builder B(I);
        B.resident.assign(I.N, 0);
        B.res_off.assign(I.N, 0);
        B.set_cuts(B.choose_cuts(S));
        B.plan(false);
        B.choose_residents(kResidentAfter);
        B.set_cuts(B.choose_cuts(S));
        B.plan(true);
        return build(I, B, true);
    };
    // Largest segment size (in value elements) whose register file fits the
    // budget: halve until it fits, then bisect between the fitting size and
    // the one above it.  If nothing fits, keep the smallest register file.
    uint64_t hi = std::max<uint64_t>(total, 1);
    Schedule best = trial(hi);
    if (best.n_regs <= reg_budget) return best;
    uint64_t lo = hi;
    bool found = false;
    while (lo > 4) {
        lo /= 2;
        Schedule c = trial(lo);
        if (c.n_regs <= reg_budget) {
            best = std::move(c);
            found = true;
            break;
        }
        if (c.n_regs < best.n_regs) best = std::move(c);
        hi = lo;
    }
    if (!found) return best;
    // invariant: lo fits, hi does not
    while (hi - lo > std::max<uint64_t>(8, lo / 16)) {
        uint64_t mid = lo + (hi - lo) / 2;
        Schedule c = trial(mid);
        if (c.n_regs <= reg_budget) {
            best = std::move(c);
            lo = mid;
        } else {
            hi = mid;
        }
    }
    return best;
}

}  // namespace ndvm
