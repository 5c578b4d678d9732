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
#include <cstdlib>
#include <cstring>
#include <map>
#include <stdexcept>
#include <string>
#include <unordered_map>

#include "slot.h"

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
    // Multiply-add fusion: fmul[c] = 1 + m when the product m is folded into
    // the sum or difference c (c reads m's operands instead of m), else 0.
    // m's value is then never formed: its only reader is c and no adjoint
    // rule reads it.  x*y + z rounds the product and then the sum, so c
    // keeps the bits of the two separate operations.
    std::vector<uint32_t> fmul;

    explicit Info(const Tape &tape) : t(tape), N(uint32_t(tape.ops.size())), P(tape.n_params) {}

    // operand values of op k (as representatives; a fused sum reads the
    // product's operands, then its other operand)
    template <class F>
    void for_operands(uint32_t k, F f) const {
        if (!fmul.empty() && fmul[k]) {
            const uint32_t m = fmul[k] - 1;
            const TapeOp &o = t.ops[k];
            f(rep[t.ops[m].a]);
            f(rep[t.ops[m].b]);
            f(rep[rep[o.a] == m ? o.b : o.a]);
            return;
        }
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

    // Fold a product into the sum or difference that is its only reader,
    // elementwise ops of one shape only (no broadcast operand).
    void fuse_products() {
        std::vector<uint32_t> readers(N, 0);
        std::vector<uint8_t> rule_reads(N, 0);
        for (uint32_t k = 0; k < N; ++k)
            if (vlive[k] && rep[k] == k) for_operands(k, [&](uint32_t s) { readers[s]++; });
        readers[rep[t.loss]]++;
        for (uint32_t k = 0; k < N; ++k)
            if (need_rev[k]) for_revreads(k, [&](uint32_t s) { rule_reads[s] = 1; });
        fmul.assign(N, 0);
        for (uint32_t c = 0; c < N; ++c) {
            const TapeOp &o = t.ops[c];
            if (!vlive[c] || rep[c] != c || kind[c] != K_COMP || (o.code != tp::ADD && o.code != tp::SUB)) continue;
            for (uint32_t side = 0; side < 2; ++side) {
                const uint32_t m = rep[side == 0 ? o.a : o.b], other = rep[side == 0 ? o.b : o.a];
                if (kind[m] != K_COMP || t.ops[m].code != tp::MUL || rep[m] != m || !vlive[m]) continue;
                if (readers[m] != 1 || rule_reads[m] || m == rep[t.loss] || m == other) continue;
                const uint32_t n = nel[c];
                if (nel[m] != n || nel[other] != n || nel[t.ops[m].a] != n || nel[t.ops[m].b] != n) continue;
                fmul[c] = m + 1;
                vlive[m] = 0;
                break;
            }
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
        fuse_products();
        last_use.assign(N, 0);
        for (uint32_t k = 0; k < N; ++k)
            if (vlive[k] && rep[k] == k) for_operands(k, [&](uint32_t s) { last_use[s] = k; });
        last_use[rep[t.loss]] = N;
        // no skippable arms unless find_arms finds them
        cone_of.assign(N, -1);
        sel_group.assign(N, -1);
        arm_of.assign(N, -1);
        hoist.assign(N, 0);
        groups.clear();
    }

    // ---- arms of numeric branches that a wave may skip (Section 6 lane
    // masking, taken per wave: when every lane of a wave decides a branch
    // the same way, the other arm's forward values and adjoint rules are not
    // run).  A group is one branch: a run of consecutive SELECT slots with the
    // same predicate operands.  Its cone on side 0 (then) / 1 (else) is the
    // set of values whose every reader is in that cone or is a select of the
    // group reading it through that side's input: values no lane needs when
    // the wave takes the other arm.  Groups inside another group's cone are
    // not skipped on their own (they are part of the outer arm).
    struct Group {
        std::vector<uint32_t> sel;       // SELECT slots, ascending
        uint32_t a = 0, b = 0;           // predicate operand slots
        std::vector<uint32_t> cone[2];   // representatives, ascending
        uint32_t lo = 0, hi = 0;         // tape range of its cones and selects
        std::vector<uint32_t> hoisted;   // observation loads laid out before the arms
    };
    std::vector<Group> groups;
    std::vector<int32_t> cone_of;        // representative -> 2 * group + side, or -1
    std::vector<int32_t> sel_group;      // SELECT slot -> group, or -1
    std::vector<int32_t> arm_of;         // slot -> 2 * group + side of the arm holding its rule, or -1
    std::vector<uint8_t> hoist;          // observation loads laid out with an earlier branch's arms

    void find_arms(uint32_t arm_min, uint32_t merge) {
        cone_of.assign(N, -1);
        sel_group.assign(N, -1);
        groups.clear();
        std::vector<uint32_t> readers(N, 0);
        for (uint32_t k = 0; k < N; ++k)
            if (vlive[k] && rep[k] == k) for_operands(k, [&](uint32_t s) { readers[s]++; });
        readers[rep[t.loss]]++;
        std::vector<Group> all;
        for (uint32_t k = 0; k < N;) {
            const TapeOp &o = t.ops[k];
            if (o.code != tp::SELECT) { ++k; continue; }
            Group g;
            g.a = o.a;
            g.b = o.b;
            uint32_t e = k;
            while (e < N && t.ops[e].code == tp::SELECT && rep[t.ops[e].a] == rep[o.a] && rep[t.ops[e].b] == rep[o.b])
                g.sel.push_back(e++);
            k = e;
            bool live = false;
            for (uint32_t q : g.sel) live = live || (vlive[q] && rep[q] == q);
            if (!live) continue;
            for (uint32_t side = 0; side < 2; ++side) {
                std::vector<uint32_t> cnt(N, 0);   // readers accounted for by the cone
                uint32_t top = 0;
                for (uint32_t q : g.sel) {
                    if (!(vlive[q] && rep[q] == q)) continue;
                    const TapeOp &so = t.ops[q];
                    const uint32_t in = rep[side == 0 ? so.c : so.d];
                    cnt[in]++;
                    top = std::max(top, in);
                }
                for (uint32_t v = top + 1; v-- > 0;) {
                    if (!cnt[v] || cnt[v] != readers[v] || rep[v] != v || !vlive[v] || kind[v] != K_COMP) continue;
                    // a select of the branch itself (one reading another) stays with the selects
                    if (std::find(g.sel.begin(), g.sel.end(), v) != g.sel.end()) continue;
                    g.cone[side].push_back(v);
                    for_operands(v, [&](uint32_t s2) { cnt[s2]++; });
                }
                std::reverse(g.cone[side].begin(), g.cone[side].end());
                // arms below arm_min elements stay unmarked
                uint32_t elems = 0;
                for (uint32_t v : g.cone[side]) elems += nel[v];
                if (elems < arm_min) g.cone[side].clear();
            }
            if (g.cone[0].empty() && g.cone[1].empty()) continue;
            all.push_back(std::move(g));
        }
        std::vector<int32_t> in_cone(N, -1);
        for (uint32_t gi = 0; gi < all.size(); ++gi)
            for (uint32_t side = 0; side < 2; ++side)
                for (uint32_t v : all[gi].cone[side]) in_cone[v] = int32_t(gi);
        std::vector<Group> kept;
        for (uint32_t gi = 0; gi < all.size(); ++gi) {
            bool nested = false;
            for (uint32_t q : all[gi].sel) nested = nested || (in_cone[rep[q]] >= 0 && in_cone[rep[q]] != int32_t(gi));
            if (!nested) kept.push_back(std::move(all[gi]));
        }
        // Branches on the same predicate value one after another (the trips
        // of a loop around a branch) share one skip test: the later arms'
        // values are computed with the first branch's, so the arms of up to
        // `merge` branches are independent chains the packer can put side
        // by side (one arm alone is mostly a dependent chain).  A later arm
        // qualifies when every value it reads from outside itself is a
        // constant, a parameter, an observation (its load moves up before
        // the skip test) or a value computed before the first branch's arm.
        hoist.assign(N, 0);
        for (size_t gi = 0; gi < kept.size();) {
            Group g = std::move(kept[gi]);
            const uint32_t at = g.sel.front();   // where the arms are laid out
            size_t e = gi + 1;
            std::vector<uint32_t> loads;
            for (uint32_t members = 1; e < kept.size() && members < merge; ++e, ++members) {
                const Group &h = kept[e];
                if (rep[h.a] != rep[g.a] || rep[h.b] != rep[g.b]) break;
                bool ok = true;
                std::vector<uint32_t> hl;
                for (uint32_t side = 0; side < 2 && ok; ++side)
                    for (uint32_t v : h.cone[side]) {
                        for_operands(v, [&](uint32_t u) {
                            if (std::binary_search(h.cone[side].begin(), h.cone[side].end(), u)) return;
                            if (kind[u] == K_CONST || kind[u] == K_PARAM) return;
                            if (kind[u] == K_OBS) {
                                if (u > at) hl.push_back(u);
                                return;
                            }
                            if (u >= at || cone_of[u] >= 0) ok = false;
                        });
                        // the arm's adjoint rules run after the first branch's
                        // select rules: every slot they add to outside the arm
                        // must have its own rule run later (lie before it)
                        const uint32_t fused = (!fmul.empty() && fmul[v]) ? fmul[v] - 1 : N;   // in the arm too
                        auto raw_ok = [&](uint32_t r) {
                            if (kind[r] != K_COMP) return;
                            if (std::binary_search(h.cone[side].begin(), h.cone[side].end(), rep[r])) return;
                            if (r >= at && r != fused) ok = false;
                        };
                        for_operands_raw(v, raw_ok);
                        if (!fmul.empty() && fmul[v]) for_operands_raw(fmul[v] - 1, raw_ok);
                    }
                if (!ok) break;
                for (uint32_t side = 0; side < 2; ++side) {
                    g.cone[side].insert(g.cone[side].end(), h.cone[side].begin(), h.cone[side].end());
                    std::sort(g.cone[side].begin(), g.cone[side].end());
                }
                g.sel.insert(g.sel.end(), h.sel.begin(), h.sel.end());
                loads.insert(loads.end(), hl.begin(), hl.end());
            }
            gi = e;
            std::sort(loads.begin(), loads.end());
            loads.erase(std::unique(loads.begin(), loads.end()), loads.end());
            for (uint32_t u : loads) hoist[u] = 1;
            g.hoisted = std::move(loads);
            const int32_t id = int32_t(groups.size());
            g.lo = g.sel.front();
            g.hi = g.sel.back();
            for (uint32_t side = 0; side < 2; ++side)
                for (uint32_t v : g.cone[side]) {
                    cone_of[v] = 2 * id + int32_t(side);
                    g.lo = std::min(g.lo, v);
                }
            for (uint32_t q : g.sel) sel_group[q] = id;
            groups.push_back(std::move(g));
        }
        // Slots whose adjoint rules lie in an arm: the cone's values; a
        // product folded into a cone value's sum (its value is never formed,
        // its rule is); duplicates of a cone value up to the branch's last
        // select (an adjoint rule there may contribute to a cone value, so it
        // must run before that value's rule).  A duplicate after the last
        // select is laid out before the arm as usual; when the wave skips the
        // arm its adjoint is exactly zero (only selects of the same predicate
        // and the arm's own values reach it), so its gated contributions are
        // nothing whatever stale values it reads.
        arm_of.assign(N, -1);
        for (uint32_t k = 0; k < N; ++k) {
            const int32_t c = cone_of[rep[k]];
            if (c >= 0 && k <= groups[uint32_t(c) / 2].hi) arm_of[k] = c;
        }
        for (uint32_t c = 0; c < N; ++c)
            if (!fmul.empty() && fmul[c] && arm_of[c] >= 0) {
                const uint32_t m = fmul[c] - 1;
                arm_of[m] = arm_of[c];
                Group &g = groups[uint32_t(arm_of[c]) / 2];
                g.lo = std::min(g.lo, m);
            }
    }
    // the cone (2 * group + side) a slot's adjoint rule or value belongs to, or -1
    int32_t cone_of_slot(uint32_t k) const { return arm_of[k]; }
};

// ------------------------------------------------------------------ allocation
struct Interval {
    uint32_t start, end, nel;
    uint32_t reg;
};

// Placement of intervals (sorted by start) into registers.  A scalar takes
// the next free register after the previous scalar's, cycling through a pool
// of `pool` registers, so that values of independent computations land in
// different registers for as long as the pool allows (immediate reuse would
// tie their micro-ops together in the packer); a block takes the first free
// run.  The file grows past the pool only when every pool register is busy.
// Without `spread`, scalars also take the first free register (the most
// compact placement).
// Returns the register high-water mark; a register whose interval ends at t
// is reusable from t + 1 on.
// Free times of the register file, with a min tree over them so that the
// first register at or after an index that is free by a given time is found
// in O(log n).  Registers past the file's end read as never free.
struct FreeTimes {
    uint32_t n = 0, cap = 1;
    std::vector<uint32_t> t{UINT32_MAX, UINT32_MAX};
    explicit FreeTimes(uint32_t pool) { resize(pool); }
    uint32_t size() const { return n; }
    uint32_t get(uint32_t i) const { return t[cap + i]; }
    void set(uint32_t i, uint32_t v) {
        i += cap;
        t[i] = v;
        for (i >>= 1; i; i >>= 1) t[i] = std::min(t[2 * i], t[2 * i + 1]);
    }
    void resize(uint32_t m) {  // new registers start free at time 0
        if (m > cap) {
            uint32_t c = cap;
            while (c < m) c *= 2;
            std::vector<uint32_t> u(2 * c, UINT32_MAX);
            for (uint32_t i = 0; i < n; ++i) u[c + i] = t[cap + i];
            cap = c;
            t.swap(u);
            for (uint32_t i = cap - 1; i; --i) t[i] = std::min(t[2 * i], t[2 * i + 1]);
        }
        for (uint32_t i = n; i < m; ++i) set(i, 0);
        n = std::max(n, m);
    }
    // first i >= lo with free time <= x, or UINT32_MAX
    uint32_t first(uint32_t lo, uint32_t x) const {
        if (lo >= n) return UINT32_MAX;
        uint32_t i = cap + lo;
        if (t[i] <= x) return lo;
        // climb until a right sibling subtree holds a candidate
        for (;;) {
            if (i == 1) return UINT32_MAX;
            if (!(i & 1) && t[i + 1] <= x) {
                i = i + 1;
                break;
            }
            i >>= 1;
        }
        while (i < cap) i = t[2 * i] <= x ? 2 * i : 2 * i + 1;
        return i - cap;
    }
};

// Returns the register high-water mark; a register whose interval ends at t
// is reusable from t + 1 on.
uint32_t allocate(std::vector<Interval> &iv, uint32_t pool, bool spread = true) {
    std::vector<uint32_t> order(iv.size());
    for (uint32_t i = 0; i < iv.size(); ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(),
                     [&](uint32_t x, uint32_t y) { return iv[x].start < iv[y].start; });
    FreeTimes busy(pool);  // first time each register is free again
    uint32_t hwm = 0, cursor = 0;
    for (uint32_t id : order) {
        Interval &v = iv[id];
        if (v.nel == 1) {
            // round robin from the cursor when spreading, else lowest free
            uint32_t r = busy.first(spread ? cursor : 0, v.start);
            if (r == UINT32_MAX && spread) r = busy.first(0, v.start);
            if (r == UINT32_MAX) {
                r = busy.size();
                busy.resize(r + 1);
            }
            busy.set(r, v.end + 1);
            v.reg = r;
            if (spread) cursor = r + 1;
            hwm = std::max(hwm, r + 1);
            continue;
        }
        // lowest run of nel registers free by the start; a run cut off by
        // the file's end is extended
        uint32_t base = busy.first(0, v.start);
        while (base != UINT32_MAX) {
            uint32_t k = 1;
            while (k < v.nel && base + k < busy.size() && busy.get(base + k) <= v.start) ++k;
            if (k == v.nel || base + k == busy.size()) break;
            base = busy.first(base + k + 1, v.start);
        }
        if (base == UINT32_MAX) base = busy.size();
        if (base + v.nel > busy.size()) busy.resize(base + v.nel);
        for (uint32_t i = 0; i < v.nel; ++i) busy.set(base + i, v.end + 1);
        v.reg = base;
        hwm = std::max(hwm, base + v.nel);
    }
    return hwm;
}

// ------------------------------------------------------------------ builder
// Abstract instruction before register assignment.
enum RIKind : uint8_t { I_LDP, I_LDC, I_CKST, I_FWD, I_STLOSS, I_ZEROP, I_SEED, I_CKLD, I_REV, I_STG,
                        I_SKIP,      // a skippable arm starts: group k, side nb, segment j
                        I_SKIPEND,   // the arm ends
                        I_ZERO };    // adjoint of slot k set to +0 (segment j): its first contribution is in a
                                     // skippable arm
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
    // save policy: values the adjoint rules read are stored in the forward
    // sweep (as segment inputs of their own segment) instead of recomputed
    bool save_reads = false;

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
                if (s >= lo && !save_reads) {
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
        // no cut inside a skippable branch: its arms are laid out next to
        // its selects, after the positions their ops had in the tape
        std::vector<uint8_t> nocut(N + 1, 0);
        for (const auto &g : I.groups)
            for (uint32_t p = g.lo + 1; p <= g.hi; ++p) nocut[p] = 1;
        std::vector<uint32_t> c{0};
        uint64_t acc = 0;
        int64_t best = -1;
        uint32_t start = 0;
        for (uint32_t k = 0; k < N; ++k) {
            if (comp_live(k)) acc += I.nel[k];
            uint32_t p = k + 1;
            if (p >= N) break;
            if (acc * 2 >= S && p > start && !nocut[p]) {
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
constexpr uint32_t kBundleWindow = 48;

// Reorder each run of forward instructions (list scheduling, earliest ready
// op first, data dependences kept) and group up to kBundleMax independent
// scalar ops of one class at one position.  The groups only order the
// abstract instructions, and with them the value intervals the registers are
// allocated from: independent ops placed side by side get distinct
// registers, which leaves the micro-op packer free to put them in one
// instruction (without this order the logistic program needs 21% more
// instructions).  Every op still computes exactly what it computed before,
// so results are unchanged bit for bit.
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

// Group scalar adjoint rules of each run of reverse instructions (for the
// same reason as the forward groups: the order of the abstract instructions
// is the order the registers are allocated in).  An op may
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

// ------------------------------------------------------------------ micro-ops
// One slot's micro-op before packing: form, flags (kUFirst), the
// immediate, and fields a, x, y, z as register numbers or indices.
constexpr uint32_t kUFirst = 1;
// a MAC whose x is a nonzero constant: the linear adjoint form (gated on x,
// which is then open) computes the same bits, so it may be packed with them
constexpr uint32_t kUAltAcc = 2;
struct UOp {
    uint32_t form, flags, imm;
    uint32_t f[4];
};

// Pseudo micro-ops that bound a skippable arm in a phase's micro-op list:
// begin carries the predicate register in f[1] and the side (0 then, 1 else)
// in imm.  They never reach the packer: each phase is packed block by block
// between them, and the encoder puts a SKIP instruction before each arm.
constexpr uint32_t kMarkBegin = 0x7FFF0001u, kMarkEnd = 0x7FFF0002u;

// index field of a checkpoint move of n rows from `row` on
uint32_t ck_row(uint32_t row, uint32_t n) {
    if (row > slot::kCkRowMask || n == 0 || n > slot::kMaxCk)
        throw std::length_error("checkpoint row beyond the index field of the device program");
    return slot::ck_field(row, n);
}

// Keys of what a micro-op reads and writes: registers r, checkpoint rows
// kKeyCkpt + row, the loss, gradient entries kKeyGrad + p.
constexpr uint64_t kKeyCkpt = 1ull << 32, kKeyLoss = 2ull << 32, kKeyGrad = 3ull << 32;

void uop_access(const UOp &u, std::vector<uint64_t> &rd, std::vector<uint64_t> &wr) {
    using namespace slot;
    rd.clear();
    wr.clear();
    const uint32_t f = u.form, im = u.imm;
    const uint32_t a = u.f[0], x = u.f[1], y = u.f[2], z = u.f[3];
    const bool acc_base = !(u.flags & kUFirst);   // adjoint forms read their target
    switch (f) {
    case MAC: case SELP: case GATEGT: case MSUB: case RSUB:
        rd = {x, y, z};
        wr = {a};
        break;
    case ACC:   // base in z: the target itself, or +0 for a first contribution
        rd = {x, y, z};
        wr = {a};
        break;
    case MACG: case ACCD: case ACCND: case ACCSEL: case ACCABS:
        rd = {x, y, z};
        if (acc_base) rd.push_back(a);
        wr = {a};
        break;
    case DOT: case DOTACC: {
        const uint32_t K = im & 31u, sa = (im >> 6) & 63u, sb = (im >> 12) & 63u;
        for (uint32_t k = 0; k < K; ++k) {
            rd.push_back(x + k * sa);
            rd.push_back(y + k * sb);
        }
        if (f == DOTACC) {
            rd.push_back(z);
            if (acc_base) rd.push_back(a);
        }
        wr = {a};
        break;
    }
    case DOTB: case DOTBACC: {
        const uint32_t K = im & 7u, N = (im >> 3) & 7u, sx = (im >> 6) & 7u, sy = (im >> 9) & 7u,
                       sc = (im >> 12) & 7u;
        for (uint32_t k = 0; k < K; ++k) {
            rd.push_back(x + k * sx);
            for (uint32_t j = 0; j < N; ++j) rd.push_back(y + k * sy + j * sc);
        }
        for (uint32_t j = 0; j < N; ++j) {
            wr.push_back(a + j);
            if (f == DOTBACC && acc_base) rd.push_back(a + j);
        }
        if (f == DOTBACC) rd.push_back(z);
        break;
    }
    case DIV: case CMPLT: case POWF:
        rd = {x, y};
        wr = {a};
        break;
    case DET2:
        rd = {x, x + 1, x + 2, x + 3};
        wr = {a};
        break;
    case NZ:
        for (uint32_t k = 0; k < im; ++k) rd.push_back(x + k);
        wr = {a};
        break;
    case SUMK:
        for (uint32_t k = 0; k < (im & 63u); ++k) rd.push_back(x + k * ((im >> 6) & 63u));
        wr = {a};
        break;
    case UN: case EXPF: case LOGCF: case LOGF: case SQRTCF: case ABSF:
        rd = {x};
        wr = {a};
        break;
    case LDOBS: case LDPARAM: case LDCONST: case ZERO:
        wr = {a};
        break;
    case CKST:
        for (uint32_t k = 0; k <= (x >> kCkRowBits); ++k) {
            rd.push_back(a + k);
            wr.push_back(kKeyCkpt + (x & kCkRowMask) + k);
        }
        break;
    case CKLD:
        for (uint32_t k = 0; k <= (x >> kCkRowBits); ++k) {
            rd.push_back(kKeyCkpt + (x & kCkRowMask) + k);
            wr.push_back(a + k);
        }
        break;
    case STLOSS:
        rd = {a};
        wr = {kKeyLoss};
        break;
    case STGRAD:
        rd = {a};
        wr = {kKeyGrad + x};
        break;
    default:
        break;
    }
}

// Instruction class of a micro-op: form and immediate must agree for
// micro-ops to share an instruction.
uint64_t uop_class(const UOp &u) { return uint64_t(u.form) | uint64_t(u.imm) << 8; }

// Pack micro-ops (in program order) into instructions of at most S slots
// by list scheduling on the dependence graph: among the next kPackWindow
// unscheduled micro-ops, each instruction takes the form (and immediate) of
// the ready one with the longest chain of dependences after it, and up to S
// ready micro-ops of that form, longest chains first, so the critical path
// of a latency-bound lane goes first.  A micro-op is ready when every value it
// reads or overwrites is final: its true and output dependences lie in
// earlier instructions, and the micro-ops that read a register it overwrites
// are scheduled (possibly in the same instruction, since every slot reads
// before any writes).  Each register and memory cell therefore sees its
// reads and writes in program order, so results are those of the sequential
// program.
constexpr uint32_t kPackWindow = 160;

std::vector<std::vector<uint32_t>> pack(std::vector<UOp> &ops, uint32_t S) {
    const uint32_t n = uint32_t(ops.size());
    // successor lists: hard (true / output dependences), soft (overwrite
    // after read)
    std::vector<uint32_t> hard_cnt(n, 0), soft_cnt(n, 0);
    std::vector<std::vector<uint32_t>> hard_succ(n), soft_succ(n);
    {
        std::unordered_map<uint64_t, uint32_t> dense;
        std::vector<int64_t> last_w;
        std::vector<std::vector<uint32_t>> readers;
        std::vector<uint64_t> rd, wr;
        auto id = [&](uint64_t key) {
            auto it = dense.emplace(key, uint32_t(last_w.size())).first;
            if (it->second == last_w.size()) {
                last_w.push_back(-1);
                readers.emplace_back();
            }
            return it->second;
        };
        std::vector<uint32_t> preds;
        for (uint32_t j = 0; j < n; ++j) {
            uop_access(ops[j], rd, wr);
            preds.clear();
            for (uint64_t r : rd) {
                const uint32_t d = id(r);
                if (last_w[d] >= 0) preds.push_back(uint32_t(last_w[d]));
            }
            for (uint64_t w : wr) {
                const uint32_t d = id(w);
                if (last_w[d] >= 0) preds.push_back(uint32_t(last_w[d]));
            }
            std::sort(preds.begin(), preds.end());
            preds.erase(std::unique(preds.begin(), preds.end()), preds.end());
            for (uint32_t p : preds) {
                hard_succ[p].push_back(j);
                hard_cnt[j]++;
            }
            preds.clear();
            for (uint64_t w : wr)
                for (uint32_t p : readers[id(w)])
                    if (p != j) preds.push_back(p);
            std::sort(preds.begin(), preds.end());
            preds.erase(std::unique(preds.begin(), preds.end()), preds.end());
            for (uint32_t p : preds) {
                soft_succ[p].push_back(j);
                soft_cnt[j]++;
            }
            for (uint64_t r : rd) readers[id(r)].push_back(j);
            for (uint64_t w : wr) {
                const uint32_t d = id(w);
                last_w[d] = j;
                readers[d].clear();
            }
        }
    }
    std::vector<uint64_t> cls(n), alt(n, ~0ull);
    for (uint32_t j = 0; j < n; ++j) {
        cls[j] = uop_class(ops[j]);
        if (ops[j].flags & kUAltAcc) alt[j] = uop_class(UOp{slot::ACC, 0, 0, {0, 0, 0, 0}});
    }
    // height: instructions from a micro-op to the end of the longest chain
    // of dependences through it (an overwrite after a read may share an
    // instruction)
    std::vector<uint32_t> height(n, 1);
    for (uint32_t j = n; j-- > 0;) {
        uint32_t h = 1;
        for (uint32_t s : hard_succ[j]) h = std::max(h, height[s] + 1);
        for (uint32_t s : soft_succ[j]) h = std::max(h, height[s]);
        height[j] = h;
    }
    std::vector<uint8_t> done(n, 0);
    std::vector<std::vector<uint32_t>> out;
    uint32_t front = 0;
    while (front < n) {
        const uint32_t end = std::min<uint32_t>(n, front + kPackWindow);
        // list scheduling by height: the class of the ready micro-op with
        // the greatest height (ties: the earliest), filled with the ready
        // micro-ops of that class in order of height; an overwrite whose
        // readers were just taken may join
        uint64_t best = 0;
        uint32_t hb = 0, top = n;
        for (uint32_t j = front; j < end; ++j) {
            if (done[j] || hard_cnt[j] || soft_cnt[j]) continue;
            if (height[j] > hb) {
                hb = height[j];
                best = cls[j];
                top = j;
            }
        }
        // a micro-op that may take either form: the one with more ready company
        if (top < n && alt[top] != ~0ull) {
            uint32_t c0 = 0, c1 = 0;
            for (uint32_t j = front; j < end; ++j) {
                if (done[j] || hard_cnt[j] || soft_cnt[j]) continue;
                c0 += cls[j] == cls[top] || alt[j] == cls[top];
                c1 += cls[j] == alt[top] || alt[j] == alt[top];
            }
            if (c1 > c0) best = alt[top];
        }
        std::vector<uint32_t> cur;
        while (cur.size() < S) {
            uint32_t pick = n;
            for (uint32_t j = front; j < end; ++j) {
                if (done[j] || (cls[j] != best && alt[j] != best) || hard_cnt[j] || soft_cnt[j]) continue;
                if (pick == n || height[j] > height[pick]) pick = j;
            }
            if (pick == n) break;
            done[pick] = 1;
            cur.push_back(pick);
            if (cls[pick] != best) ops[pick].form = slot::ACC;   // the alternative form
            for (uint32_t s : soft_succ[pick]) soft_cnt[s]--;
        }
        for (uint32_t j : cur)
            for (uint32_t s : hard_succ[j]) hard_cnt[s]--;
        out.push_back(std::move(cur));
        while (front < n && done[front]) ++front;
    }
    return out;
}

// Micro-op emitter of one program: registers named by the scheduler, plus a
// rotating pool of temporaries for values that live inside one op's
// lowering (predicates, node gates, partial products, 2x2 inverses).
struct UEmit {
    std::vector<UOp> ops;
    uint32_t tmp0 = 0, n_tmp = 0, next_tmp = 0;
    void put(uint32_t form, uint32_t a, uint32_t flags, uint32_t x = 0, uint32_t y = 0, uint32_t z = 0,
             uint32_t imm = 0) {
        if (imm > slot::kMaxImm) throw std::length_error("immediate beyond the header field of the device program");
        ops.push_back({form, flags, imm, {a, x, y, z}});
    }
    uint32_t used_tmp = 0;   // temporaries touched (0 when the program needs none)
    // a block of n consecutive temporaries
    uint32_t tmp(uint32_t n = 1) {
        if (next_tmp + n > n_tmp) next_tmp = 0;
        const uint32_t r = tmp0 + next_tmp;
        next_tmp += n;
        used_tmp = std::max(used_tmp, next_tmp);
        return r;
    }
};

constexpr uint32_t kTemps = 24;

// Build the forward phase (shared by both programs) and, for the gradient
// program, the reverse phase; returns the slot program with registers
// assigned and micro-ops packed S to an instruction.
// Without `full`, stops once the registers are known (n_regs,
// n_temps_used and the counts of the lowering): what the search over
// segment sizes needs, without packing and encoding.
Schedule build(const Info &I, Builder &B, bool with_grad, uint32_t S, uint32_t reg_budget, uint32_t n_temps,
               bool full) {
    using namespace slot;
    const Tape &t = I.t;
    const uint32_t N = I.N, P = I.P;
    // static registers: param values, param adjoints, sinks for results of
    // unused slots, the constant pool, residents.  The pool holds the tape's
    // constants, then 1, -1, -0, 2, the clamp threshold 1e-8 and +0.
    const uint32_t nt = uint32_t(t.consts.size()), nc = nt + 6;
    const uint32_t kSink = 2 * P, kConst0 = 2 * P + kMaxBlock;
    const uint32_t kOne = kConst0 + nt, kMinusOne = kOne + 1, kNegZero = kOne + 2, kTwo = kOne + 3,
                   kEps = kOne + 4, kZeroC = kOne + 5;
    const uint32_t kStatic = kConst0 + nc + B.res_elems;
    // registers the value allocation may spread over: the budget less the
    // static registers and the temporaries
    const uint32_t pool = reg_budget > kStatic + n_temps ? reg_budget - kStatic - n_temps : 1;
    const uint32_t m = uint32_t(B.cuts.size());
    Schedule Sch;
    Sch.slots = S;
    Sch.n_segments = with_grad ? m : 1;
    Sch.static_regs = kStatic;
    Sch.consts = t.consts;
    for (double v : {1.0, -1.0, -0.0, 2.0, 1e-8, 0.0}) Sch.consts.push_back(v);

    // ---- forward phase: abstract instructions + value intervals
    std::vector<AI> fa;
    std::vector<uint32_t> ckrow_base(m + 1, 0);
    if (with_grad) {
        uint32_t row = 0;
        for (uint32_t j = 0; j < m; ++j) {
            ckrow_base[j] = row;
            for (uint32_t s : B.livein[j]) row += I.nel[s];
        }
        ckrow_base[m] = row;
        Sch.n_ckpt_rows = row;
    }
    for (uint32_t p = 0; p < P; ++p) fa.push_back({I_LDP, p, 0});
    fa.push_back({I_LDC, 0, nc});
    uint32_t next_cut = 1;
    for (uint32_t k = 0; k < N; ++k) {
        if (with_grad && !B.save_reads) {
            while (next_cut < m && B.cuts[next_cut] == k) {
                for (uint32_t i = 0; i < B.livein[next_cut].size(); ++i) fa.push_back({I_CKST, next_cut, i});
                ++next_cut;
            }
        }
        if (I.cone_of_slot(k) >= 0 && B.comp_live(k)) continue;   // laid out with its branch's selects
        if (I.hoist[k]) continue;                                  // loaded before an earlier branch's arms
        if (I.sel_group[k] >= 0 && I.groups[uint32_t(I.sel_group[k])].sel.front() == k) {
            // the branch's arms, each behind a skip test: its cone's values
            // in tape order, right before the selects (the observations the
            // arms of later branches on the same predicate read first)
            const uint32_t gi = uint32_t(I.sel_group[k]);
            for (uint32_t u : I.groups[gi].hoisted) fa.push_back({I_FWD, u, 0});
            for (uint8_t side = 0; side < 2; ++side) {
                if (I.groups[gi].cone[side].empty()) continue;
                AI sk{I_SKIP, gi, 0};
                sk.nb = side;
                fa.push_back(sk);
                for (uint32_t v : I.groups[gi].cone[side]) fa.push_back({I_FWD, v, 0});
                fa.push_back({I_SKIPEND, gi, 0});
            }
        }
        if (B.comp_live(k) || (I.kind[k] == K_OBS && I.vlive[k])) fa.push_back({I_FWD, k, 0});
    }
    fa.push_back({I_STLOSS, t.loss, 0});
    fa = bundle_forward(I, fa);
    if (with_grad && B.save_reads) {
        // save policy: every stored value is stored right after the forward
        // instruction that computes it, so no value stays live for its store
        std::unordered_map<uint32_t, std::vector<std::pair<uint32_t, uint32_t>>> saves_of;
        for (uint32_t j = 0; j < m; ++j)
            for (uint32_t i = 0; i < B.livein[j].size(); ++i) saves_of[B.livein[j][i]].push_back({j, i});
        std::vector<AI> out;
        out.reserve(fa.size() + saves_of.size());
        for (const AI &a : fa) {
            out.push_back(a);
            if (a.kind != I_FWD) continue;
            for (uint32_t b = 0; b < a.nops(); ++b) {
                auto it = saves_of.find(a.op(b));
                if (it == saves_of.end()) continue;
                for (const auto &ji : it->second) out.push_back({I_CKST, ji.first, ji.second});
            }
        }
        fa = std::move(out);
    }
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
        } else if (a.kind == I_SKIP) {
            use(I.rep[I.groups[a.k].a]);
            use(I.rep[I.groups[a.k].b]);
        }
    }
    // spread over the pool; compact when that does not fit (blocks need
    // contiguous free registers, which spreading fragments)
    uint32_t fhwm = allocate(fiv, pool);
    if (fhwm > pool) fhwm = allocate(fiv, 0, false);
    Sch.fwd_regs = fhwm;

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

    UEmit E;
    E.tmp0 = kStatic + fhwm;   // forward temporaries above the forward registers
    E.n_tmp = n_temps;
    // x*y + z.  When a multiplier is a nonzero constant it goes to x and the
    // micro-op is marked kUAltAcc: the linear adjoint form computes the same
    // bits then (its gate, that constant, is open; the product and the sum
    // commute), so the packer may place it among adjoint rules.
    auto nz_const = [&](uint32_t s) {
        s = I.rep[s];
        return I.kind[s] == K_CONST && t.consts[t.ops[s].imm] != 0.0;
    };
    auto put_mac = [&](uint32_t d, uint32_t x, uint32_t y, uint32_t z, bool xc, bool yc) {
        if (xc || yc)
            E.put(MAC, d, kUAltAcc, xc ? x : y, xc ? y : x, z);
        else
            E.put(MAC, d, 0, x, y, z);
    };
    auto mov = [&](uint32_t d, uint32_t x) { put_mac(d, x, kOne, kNegZero, false, true); };

    // forward computation of op k into dst (registers from `operand`)
    auto emit_fwd = [&](uint32_t k, auto operand, uint32_t dst) {
        const TapeOp &o = t.ops[k];
        const uint32_t n = I.nel[k];
        switch (o.code) {
        case tp::OBS:
            E.put(LDOBS, dst, 0, o.imm);
            return;
        case tp::ADD: case tp::SUB: case tp::MUL: case tp::DIV: {
            if (I.fmul[k]) {   // product folded in: x*y + z, x*y - z or z - x*y
                const uint32_t mm = I.fmul[k] - 1;
                const bool m_first = I.rep[o.a] == mm;
                const uint32_t X = operand(t.ops[mm].a), Y = operand(t.ops[mm].b), Z = operand(m_first ? o.b : o.a);
                if (o.code == tp::ADD) {
                    const bool xc = nz_const(t.ops[mm].a), yc = nz_const(t.ops[mm].b);
                    for (uint32_t i = 0; i < n; ++i) put_mac(dst + i, X + i, Y + i, Z + i, xc, yc);
                    return;
                }
                const uint32_t f = m_first ? MSUB : RSUB;
                for (uint32_t i = 0; i < n; ++i) E.put(f, dst + i, 0, X + i, Y + i, Z + i);
                return;
            }
            const uint32_t A = operand(o.a), Bv = operand(o.b);
            const bool as = I.nel[o.a] == 1 && n > 1, bs = I.nel[o.b] == 1 && n > 1;
            for (uint32_t i = 0; i < n; ++i) {
                const uint32_t xa = as ? A : A + i, xb = bs ? Bv : Bv + i;
                switch (o.code) {
                case tp::ADD: put_mac(dst + i, xa, kOne, xb, false, true); break;
                case tp::SUB: put_mac(dst + i, xb, kMinusOne, xa, false, true); break;
                case tp::MUL: put_mac(dst + i, xa, xb, kNegZero, nz_const(o.a), nz_const(o.b)); break;
                default: E.put(DIV, dst + i, 0, xa, xb); break;
                }
            }
            return;
        }
        case tp::NEG: {
            const uint32_t A = operand(o.a);
            for (uint32_t i = 0; i < n; ++i) put_mac(dst + i, A + i, kMinusOne, kNegZero, false, true);
            return;
        }
        case tp::EXP: case tp::LOG: case tp::SQRT: case tp::ABS: {
            const uint32_t A = operand(o.a);
            const uint32_t f = o.code == tp::EXP ? EXPF : o.code == tp::LOG ? LOGCF : o.code == tp::SQRT ? SQRTCF : ABSF;
            for (uint32_t i = 0; i < n; ++i) E.put(f, dst + i, 0, A + i);
            return;
        }
        case tp::SIN: case tp::COS: {
            const uint32_t A = operand(o.a);
            for (uint32_t i = 0; i < n; ++i) E.put(UN, dst + i, 0, A + i, 0, 0, o.code == tp::SIN ? U_SIN : U_COS);
            return;
        }
        case tp::POW:
            E.put(POWF, dst, 0, operand(o.a), operand(o.b));
            return;
        case tp::DOT:
            E.put(DOT, dst, 0, operand(o.a), operand(o.b), 0, dot_imm(I.nel[o.a], 1, 1, false));
            return;
        case tp::MATMUL: {   // one block of q outputs per row
            const uint32_t A = operand(o.a), Bv = operand(o.b);
            const uint32_t mm = t.ops[o.a].rows, kk = t.ops[o.a].cols, q = t.ops[o.b].cols;
            for (uint32_t i = 0; i < mm; ++i)
                E.put(DOTB, dst + i * q, 0, A + i * kk, Bv, 0, dotb_imm(kk, q, 1, q, 1, false));
            return;
        }
        case tp::TRANSPOSE: {
            const uint32_t A = operand(o.a), mm = t.ops[o.a].rows, q = t.ops[o.a].cols;
            for (uint32_t i = 0; i < mm; ++i)
                for (uint32_t j = 0; j < q; ++j) mov(dst + j * mm + i, A + i * q + j);
            return;
        }
        case tp::TRACE: {
            const uint32_t sz = t.ops[o.a].rows;
            E.put(SUMK, dst, 0, operand(o.a), 0, 0, sz | (sz + 1) << 6);
            return;
        }
        case tp::INV: {
            const uint32_t A = operand(o.a), sz = t.ops[o.a].rows;
            if (sz == 1) {
                E.put(DIV, dst, 0, kOne, A);
                return;
            }
            // adjugate times r = 1 / det; (-a) * r is computed as a * (-r),
            // the same bits
            const uint32_t d = E.tmp(), r = E.tmp(), nr = E.tmp();
            E.put(DET2, d, 0, A);
            E.put(DIV, r, 0, kOne, d);
            put_mac(nr, r, kMinusOne, kNegZero, false, true);
            E.put(MAC, dst + 0, 0, A + 3, r, kNegZero);
            E.put(MAC, dst + 1, 0, A + 1, nr, kNegZero);
            E.put(MAC, dst + 2, 0, A + 2, nr, kNegZero);
            E.put(MAC, dst + 3, 0, A + 0, r, kNegZero);
            return;
        }
        case tp::DET: case tp::LOGDET: {
            const uint32_t A = operand(o.a), sz = t.ops[o.a].rows;
            uint32_t d = A;
            if (sz == 2) {
                d = o.code == tp::DET ? dst : E.tmp();
                E.put(DET2, d, 0, A);
            } else if (o.code == tp::DET) {
                mov(dst, A);
            }
            if (o.code == tp::LOGDET) E.put(LOGCF, dst, 0, d);
            return;
        }
        case tp::OUTER: {
            const uint32_t A = operand(o.a), Bv = operand(o.b);
            const uint32_t mm = t.ops[o.a].rows, q = t.ops[o.b].rows;
            for (uint32_t i = 0; i < mm; ++i)
                for (uint32_t j = 0; j < q; ++j) E.put(MAC, dst + i * q + j, 0, A + i, Bv + j, kNegZero);
            return;
        }
        case tp::PACK:
            for (uint32_t i = 0; i < o.b; ++i) mov(dst + i, operand(t.aux[o.a + i]));
            return;
        case tp::INDEX:
            mov(dst, operand(o.a) + o.imm);
            return;
        case tp::SELECT: {
            const uint32_t p = E.tmp();
            E.put(CMPLT, p, 0, operand(o.a), operand(o.b));
            const uint32_t C = operand(o.c), D = operand(o.d);
            for (uint32_t i = 0; i < n; ++i) E.put(SELP, dst + i, 0, p, C + i, D + i);
            return;
        }
        default:
            throw std::logic_error("unknown tape op in the scheduler");
        }
    };

    for (const AI &a : fa) {
        switch (a.kind) {
        case I_LDP: E.put(LDPARAM, a.k, 0, a.k); break;
        case I_LDC:
            for (uint32_t i = 0; i < a.j; ++i) E.put(LDCONST, kConst0 + i, 0, i);
            break;
        case I_CKST: {
            const uint32_t s = B.livein[a.k][a.j];
            uint32_t row = ckrow_base[a.k];
            for (uint32_t i = 0; i < a.j; ++i) row += I.nel[B.livein[a.k][i]];
            const uint32_t src = fwd_operand(s);
            for (uint32_t e = 0; e < I.nel[s]; e += kMaxCk)
                E.put(CKST, src + e, 0, ck_row(row + e, std::min(kMaxCk, I.nel[s] - e)));
            Sch.ckpt_elems_stored += I.nel[s];
            break;
        }
        case I_FWD:
            for (uint32_t b = 0; b < a.nops(); ++b) emit_fwd(a.op(b), fwd_operand, fwd_operand(a.op(b)));
            Sch.n_fwd_ops += a.nops();
            break;
        case I_STLOSS: E.put(STLOSS, fwd_operand(a.k), 0); break;
        case I_SKIP: {   // predicate of the branch, then the arm's opening mark
            const auto &g = I.groups[a.k];
            const uint32_t pt = E.tmp();
            E.put(CMPLT, pt, 0, fwd_operand(g.a), fwd_operand(g.b));
            E.ops.push_back({kMarkBegin, 0, a.nb, {0, pt, 0, 0}});
            break;
        }
        case I_SKIPEND: E.ops.push_back({kMarkEnd, 0, 0, {0, 0, 0, 0}}); break;
        }
    }
    std::vector<UOp> fwd_ops;
    uint32_t rhwm = 0;
    Sch.n_regs = kStatic + fhwm + E.used_tmp;
    Sch.n_temps_used = E.used_tmp;
    if (with_grad) {
        fwd_ops = std::move(E.ops);
        E.ops.clear();
    }

    if (with_grad) {
        // ---- reverse phase
        std::vector<AI> ra;
        ra.push_back({I_ZEROP, 0, 0});
        ra.push_back({I_SEED, t.loss, 0});
        // Checkpoint restores wait for HBM inside their instruction, so the
        // restores of consecutive segments are issued together when their
        // moves fit one instruction (S slots): the later segments' values
        // then wait in registers while the earlier segment runs.
        auto ck_moves = [&](uint32_t j) {
            uint32_t n = 0;
            for (uint32_t s : B.livein[j]) n += (I.nel[s] + kMaxCk - 1) / kMaxCk;
            return n;
        };
        std::vector<uint8_t> restored(m, 0);
        // adjoints whose first contribution has been laid out (the first
        // contribution stores instead of adding)
        std::vector<uint8_t> touched_sim(N, 0);
        auto mark_touched = [&](uint32_t k) {
            I.for_targets(k, [&](uint32_t tg) {
                if (I.kind[tg] == K_COMP && I.active[tg]) touched_sim[tg] = 1;
            });
        };
        if (I.kind[t.loss] == K_COMP) touched_sim[t.loss] = 1;
        for (uint32_t j = m; j-- > 0;) {
            if (!restored[j]) {
                uint32_t moves = ck_moves(j), last = j;
                while (last > 0 && moves + ck_moves(last - 1) <= S && ck_moves(last - 1) > 0) moves += ck_moves(--last);
                for (uint32_t q = j + 1; q-- > last;) {
                    for (uint32_t i = 0; i < B.livein[q].size(); ++i) ra.push_back({I_CKLD, q, i});
                    restored[q] = 1;
                }
            }
            for (uint32_t s : B.recomp[j]) ra.push_back({I_FWD, s, j});
            // position of each branch's last select rule in this segment
            std::unordered_map<int32_t, uint32_t> last_sel;
            for (uint32_t qi = 0; qi < B.revops[j].size(); ++qi)
                if (I.sel_group[B.revops[j][qi]] >= 0) last_sel[I.sel_group[B.revops[j][qi]]] = qi;
            for (uint32_t qi = 0; qi < B.revops[j].size(); ++qi) {
                const uint32_t k = B.revops[j][qi];
                if (I.cone_of_slot(k) >= 0) continue;   // applied in its arm, after the branch's selects
                ra.push_back({I_REV, k, j});
                mark_touched(k);
                const int32_t gsel = I.sel_group[k];
                if (gsel < 0) continue;
                // after the branch's last select rule: each arm's rules behind a
                // skip test (descending slot order, as in the tape's reverse;
                // with several branches on one predicate, after the last
                // select rule of the first)
                const uint32_t gi = uint32_t(gsel);
                if (last_sel.at(gsel) != qi) continue;
                for (uint8_t side = 2; side-- > 0;) {
                    std::vector<uint32_t> arm;   // the segment's rules of the arm, descending
                    for (uint32_t q = 0; q < B.revops[j].size(); ++q)
                        if (I.cone_of_slot(B.revops[j][q]) == int32_t(2 * gi + side)) arm.push_back(B.revops[j][q]);
                    if (arm.empty()) continue;
                    // an adjoint outside the arm whose first contribution the arm
                    // would make starts at +0 before the arm instead
                    for (uint32_t r : arm)
                        I.for_targets(r, [&](uint32_t tg) {
                            if (I.kind[tg] != K_COMP || !I.active[tg] || touched_sim[tg]) return;
                            if (I.cone_of_slot(tg) == int32_t(2 * gi + side)) return;
                            ra.push_back({I_ZERO, tg, j});
                            touched_sim[tg] = 1;
                        });
                    AI sk{I_SKIP, gi, j};
                    sk.nb = side;
                    ra.push_back(sk);
                    for (uint32_t r : arm) {
                        ra.push_back({I_REV, r, j});
                        mark_touched(r);
                    }
                    ra.push_back({I_SKIPEND, gi, j});
                }
            }
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
                const uint32_t s = B.livein[a.k][a.j];
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
            case I_REV:
                for (uint32_t b = 0; b < a.nops(); ++b) {
                    const uint32_t k = a.op(b);
                    I.for_revreads(k, [&](uint32_t s) { vuse(s, a.j, ti); });
                    I.for_targets(k, [&](uint32_t s) { contrib(s, ti); });
                    const int32_t g = adj_of[k];
                    if (g < 0) throw std::logic_error("adjoint rule laid out before any contribution to it");
                    riv[g].end = std::max(riv[g].end, ti);
                }
                break;
            case I_ZERO:
                contrib(a.k, ti);
                break;
            case I_SKIP:
                vuse(I.rep[I.groups[a.k].a], a.j, ti);
                vuse(I.rep[I.groups[a.k].b], a.j, ti);
                break;
            default:
                break;
            }
        }
        rhwm = allocate(riv, pool);
        if (rhwm > pool) rhwm = allocate(riv, 0, false);
        Sch.rev_regs = rhwm;

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
        // adjoint register of a target and whether this is its first
        // contribution; kNone when the target has no adjoint
        constexpr uint32_t kNone = 0xFFFFFFFFu;
        auto target = [&](uint32_t s, uint32_t *flags) -> uint32_t {
            *flags = 0;
            if (I.kind[s] == K_PARAM) return P + t.ops[s].imm;
            if (I.kind[s] != K_COMP || !I.active[s]) return kNone;
            const uint32_t r = kStatic + riv[adj_of[s]].reg;
            if (!touched[s]) {
                touched[s] = 1;
                *flags = kUFirst;
            }
            return r;
        };
        auto adjreg = [&](uint32_t s) { return kStatic + riv[adj_of[s]].reg; };

        E.tmp0 = kStatic + std::max(fhwm, rhwm);
        E.n_tmp = n_temps;
        E.next_tmp = 0;
        E.used_tmp = 0;

        // adjoint rule of op k (Appendix C, table tab:adjoints)
        auto emit_rev = [&](uint32_t k, uint32_t j) {
            const TapeOp &o = t.ops[k];
            const uint32_t n = I.nel[k];
            const uint32_t g = adjreg(k);
            auto v = [&](uint32_t s) { return rev_operand(s, j); };
            Sch.n_rev_ops++;
            // gate of the node: its adjoint itself when scalar, else a flag
            // register set when any element is nonzero
            uint32_t gate = g;
            auto node_gate = [&](uint32_t nel) {
                if (nel > 1) {
                    gate = E.tmp();
                    E.put(NZ, gate, 0, g, 0, 0, nel);
                } else {
                    gate = g;
                }
            };
            // t += x * y under the node gate
            auto acc = [&](uint32_t tr, uint32_t fl, uint32_t x, uint32_t y) {
                if (tr == kNone) return;
                if (gate == x)
                    E.put(ACC, tr, 0, x, y, (fl & kUFirst) ? kZeroC : tr);
                else
                    E.put(MACG, tr, fl, x, y, gate);
            };
            uint32_t fa_ = 0, fb_ = 0;
            switch (o.code) {
            case tp::ADD: case tp::SUB: {
                node_gate(n);
                const uint32_t ta = target(o.a, &fa_);
                for (uint32_t i = 0; i < n; ++i) acc(ta == kNone ? kNone : ta + i, fa_, g + i, kOne);
                const uint32_t tb = target(o.b, &fb_);
                for (uint32_t i = 0; i < n; ++i)
                    acc(tb == kNone ? kNone : tb + i, fb_, g + i, o.code == tp::ADD ? kOne : kMinusOne);
                return;
            }
            case tp::MUL: {
                node_gate(n);
                const uint32_t A = v(o.a), Bv = v(o.b);
                const bool as = I.nel[o.a] == 1 && n > 1, bs = I.nel[o.b] == 1 && n > 1;
                const uint32_t ta = target(o.a, &fa_);
                if (as) {   // z = s * M: ds = sum_i g_i M_i
                    if (ta != kNone) E.put(DOTACC, ta, fa_, g, Bv, gate, dot_imm(n, 1, 1, false));
                } else {
                    for (uint32_t i = 0; i < n; ++i) acc(ta == kNone ? kNone : ta + i, fa_, g + i, bs ? Bv : Bv + i);
                }
                const uint32_t tb = target(o.b, &fb_);
                if (bs) {   // z = M * s
                    if (tb != kNone) E.put(DOTACC, tb, fb_, g, A, gate, dot_imm(n, 1, 1, false));
                } else {
                    for (uint32_t i = 0; i < n; ++i) acc(tb == kNone ? kNone : tb + i, fb_, g + i, as ? A : A + i);
                }
                return;
            }
            case tp::DIV: {
                node_gate(n);
                const uint32_t Bv = v(o.b), Z = v(k);
                const bool bs = I.nel[o.b] == 1 && n > 1;
                const uint32_t ta = target(o.a, &fa_);
                if (ta != kNone)
                    for (uint32_t i = 0; i < n; ++i) E.put(ACCD, ta + i, fa_, g + i, bs ? Bv : Bv + i, gate);
                const uint32_t tb = target(o.b, &fb_);
                if (tb != kNone) {
                    if (bs) {   // z = M / s: ds -= (sum_i g_i z_i) / s
                        const uint32_t s = E.tmp();
                        E.put(DOT, s, 0, g, Z, 0, dot_imm(n, 1, 1, false));
                        E.put(ACCND, tb, fb_, s, Bv, gate);
                    } else {
                        for (uint32_t i = 0; i < n; ++i) {
                            const uint32_t gz = E.tmp();
                            E.put(MAC, gz, 0, g + i, Z + i, kNegZero);
                            E.put(ACCND, tb + i, fb_, gz, Bv + i, gate);
                        }
                    }
                }
                return;
            }
            case tp::NEG: case tp::EXP: case tp::LOG: case tp::SQRT: case tp::SIN: case tp::COS: case tp::ABS: {
                node_gate(n);
                const uint32_t ta = target(o.a, &fa_);
                if (ta == kNone) return;
                for (uint32_t i = 0; i < n; ++i) {
                    const uint32_t tr = ta + i, gi = g + i;
                    switch (o.code) {
                    case tp::NEG: acc(tr, fa_, gi, kMinusOne); break;
                    case tp::EXP: acc(tr, fa_, gi, v(k) + i); break;
                    case tp::LOG: {
                        const uint32_t fl = E.tmp();
                        E.put(GATEGT, fl, 0, v(o.a) + i, kEps, gate);
                        E.put(ACCD, tr, fa_, gi, v(o.a) + i, fl);
                        break;
                    }
                    case tp::SQRT: {
                        const uint32_t tz = E.tmp(), fl = E.tmp();
                        put_mac(tz, kTwo, v(k) + i, kNegZero, true, false);
                        E.put(GATEGT, fl, 0, v(o.a) + i, kEps, gate);
                        E.put(ACCD, tr, fa_, gi, tz, fl);
                        break;
                    }
                    case tp::SIN: {
                        const uint32_t c = E.tmp();
                        E.put(UN, c, 0, v(o.a) + i, 0, 0, U_COS);
                        acc(tr, fa_, gi, c);
                        break;
                    }
                    case tp::COS: {
                        const uint32_t s = E.tmp(), ns = E.tmp();
                        E.put(UN, s, 0, v(o.a) + i, 0, 0, U_SIN);
                        put_mac(ns, s, kMinusOne, kNegZero, false, true);
                        acc(tr, fa_, gi, ns);
                        break;
                    }
                    default:
                        E.put(ACCABS, tr, fa_, gi, v(o.a) + i, gate);
                        break;
                    }
                }
                return;
            }
            case tp::POW: {
                const uint32_t A = v(o.a), Bv = v(o.b), Z = v(k);
                const uint32_t ta = target(o.a, &fa_);
                if (ta != kNone) {   // a += ((g * b) * z) / a
                    const uint32_t t1 = E.tmp(), t2 = E.tmp();
                    E.put(MAC, t1, 0, g, Bv, kNegZero);
                    E.put(MAC, t2, 0, t1, Z, kNegZero);
                    E.put(ACCD, ta, fa_, t2, A, g);
                }
                const uint32_t tb = target(o.b, &fb_);
                if (tb != kNone) {   // b += (g * z) * ln a
                    const uint32_t t3 = E.tmp(), t4 = E.tmp();
                    E.put(MAC, t3, 0, g, Z, kNegZero);
                    E.put(LOGF, t4, 0, A);
                    E.put(MACG, tb, fb_, t3, t4, g);
                }
                return;
            }
            case tp::DOT: {
                gate = g;
                const uint32_t A = v(o.a), Bv = v(o.b), ne = I.nel[o.a];
                const uint32_t ta = target(o.a, &fa_);
                if (ta != kNone)
                    for (uint32_t i = 0; i < ne; ++i) acc(ta + i, fa_, g, Bv + i);
                const uint32_t tb = target(o.b, &fb_);
                if (tb != kNone)
                    for (uint32_t i = 0; i < ne; ++i) acc(tb + i, fb_, g, A + i);
                return;
            }
            case tp::MATMUL: {
                const uint32_t A = v(o.a), Bv = v(o.b);
                const uint32_t mm = t.ops[o.a].rows, kk = t.ops[o.a].cols, q = t.ops[o.b].cols;
                node_gate(mm * q);
                // dA[i, p] = sum_j G[i, j] B[p, j]: a block over p per row i
                const uint32_t ta = target(o.a, &fa_);
                if (ta != kNone)
                    for (uint32_t i = 0; i < mm; ++i)
                        E.put(DOTBACC, ta + i * kk, fa_, g + i * q, Bv, gate, dotb_imm(q, kk, 1, 1, q, false));
                // dB[p, j] = sum_i A[i, p] G[i, j]: a block over j per row p
                const uint32_t tb = target(o.b, &fb_);
                if (tb != kNone)
                    for (uint32_t p = 0; p < kk; ++p)
                        E.put(DOTBACC, tb + p * q, fb_, A + p, g, gate, dotb_imm(mm, q, kk, q, 1, false));
                return;
            }
            case tp::OUTER: {
                const uint32_t A = v(o.a), Bv = v(o.b);
                const uint32_t mm = t.ops[o.a].rows, q = t.ops[o.b].rows;
                node_gate(mm * q);
                const uint32_t ta = target(o.a, &fa_);
                if (ta != kNone)
                    for (uint32_t i = 0; i < mm; ++i) E.put(DOTACC, ta + i, fa_, g + i * q, Bv, gate, dot_imm(q, 1, 1, false));
                const uint32_t tb = target(o.b, &fb_);
                if (tb != kNone)
                    for (uint32_t jj = 0; jj < q; ++jj) E.put(DOTACC, tb + jj, fb_, g + jj, A, gate, dot_imm(mm, q, 1, false));
                return;
            }
            case tp::TRANSPOSE: {
                const uint32_t mm = t.ops[o.a].rows, q = t.ops[o.a].cols;
                node_gate(n);
                const uint32_t ta = target(o.a, &fa_);
                if (ta != kNone)
                    for (uint32_t i = 0; i < mm; ++i)
                        for (uint32_t jj = 0; jj < q; ++jj) E.put(MACG, ta + i * q + jj, fa_, g + jj * mm + i, kOne, gate);
                return;
            }
            case tp::TRACE: {
                gate = g;
                const uint32_t sz = t.ops[o.a].rows;
                const uint32_t ta = target(o.a, &fa_);
                if (ta == kNone) return;
                for (uint32_t i = 0; i < sz; ++i)
                    for (uint32_t jj = 0; jj < sz; ++jj) {
                        if (i == jj)
                            acc(ta + i * sz + jj, fa_, g, kOne);
                        else if (fa_ & kUFirst)
                            E.put(ZERO, ta + i * sz + jj, 0);
                    }
                return;
            }
            case tp::INV: {
                const uint32_t sz = t.ops[o.a].rows, Z = v(k);
                node_gate(sz * sz);
                const uint32_t ta = target(o.a, &fa_);
                if (ta == kNone) return;
                // M1 = B^T G, then A -= M1 B^T  (B the inverse)
                const uint32_t M1 = E.tmp(sz * sz);
                for (uint32_t i = 0; i < sz; ++i)
                    for (uint32_t jj = 0; jj < sz; ++jj) E.put(DOT, M1 + i * sz + jj, 0, Z + i, g + jj, 0, dot_imm(sz, sz, sz, false));
                for (uint32_t i = 0; i < sz; ++i)
                    for (uint32_t jj = 0; jj < sz; ++jj)
                        E.put(DOTACC, ta + i * sz + jj, fa_, M1 + i * sz, Z + jj * sz, gate, dot_imm(sz, 1, 1, true));
                return;
            }
            case tp::DET: case tp::LOGDET: {
                const uint32_t A = v(o.a), sz = t.ops[o.a].rows;
                const uint32_t ta = target(o.a, &fa_);
                if (ta == kNone) return;
                // the inverse of A, recomputed as in the forward op
                const uint32_t Ai = E.tmp(sz * sz);
                if (sz == 1) {
                    E.put(DIV, Ai, 0, kOne, A);
                } else {
                    const uint32_t d = E.tmp(), r = E.tmp(), nr = E.tmp();
                    E.put(DET2, d, 0, A);
                    E.put(DIV, r, 0, kOne, d);
                    put_mac(nr, r, kMinusOne, kNegZero, false, true);
                    E.put(MAC, Ai + 0, 0, A + 3, r, kNegZero);
                    E.put(MAC, Ai + 1, 0, A + 1, nr, kNegZero);
                    E.put(MAC, Ai + 2, 0, A + 2, nr, kNegZero);
                    E.put(MAC, Ai + 3, 0, A + 0, r, kNegZero);
                }
                uint32_t scale = g, on = g;
                if (o.code == tp::DET) {   // d det / dA = det * A^-T
                    scale = E.tmp();
                    E.put(MAC, scale, 0, g, v(k), kNegZero);
                } else {                   // d log det / dA = A^-T where det > 1e-8
                    uint32_t d = A;
                    if (sz == 2) {
                        d = E.tmp();
                        E.put(DET2, d, 0, A);
                    }
                    on = E.tmp();
                    E.put(GATEGT, on, 0, d, kEps, g);
                }
                for (uint32_t i = 0; i < sz; ++i)
                    for (uint32_t jj = 0; jj < sz; ++jj) E.put(MACG, ta + i * sz + jj, fa_, scale, Ai + jj * sz + i, on);
                return;
            }
            case tp::PACK: {
                node_gate(n);
                for (uint32_t i = 0; i < o.b; ++i) {
                    uint32_t fl;
                    const uint32_t tr = target(t.aux[o.a + i], &fl);
                    if (tr != kNone) E.put(MACG, tr, fl, g + i, kOne, gate);
                }
                return;
            }
            case tp::INDEX: {
                gate = g;
                const uint32_t ne = I.nel[o.a];
                const uint32_t ta = target(o.a, &fa_);
                if (ta == kNone) return;
                if (fa_ & kUFirst)
                    for (uint32_t i = 0; i < ne; ++i)
                        if (i != o.imm) E.put(ZERO, ta + i, 0);
                acc(ta + o.imm, fa_, g, kOne);
                return;
            }
            case tp::SELECT: {
                node_gate(n);
                const uint32_t p = E.tmp();
                E.put(CMPLT, p, 0, v(o.a), v(o.b));
                const uint32_t tc = target(o.c, &fa_);
                if (tc != kNone)
                    for (uint32_t i = 0; i < n; ++i) E.put(ACCSEL, tc + i, fa_, g + i, p, gate, 1);
                const uint32_t td = target(o.d, &fb_);
                if (td != kNone)
                    for (uint32_t i = 0; i < n; ++i) E.put(ACCSEL, td + i, fb_, g + i, p, gate, 0);
                return;
            }
            default:
                throw std::logic_error("unknown tape op in the reverse scheduler");
            }
        };

        for (const AI &a : ra) {
            switch (a.kind) {
            case I_ZEROP:
                for (uint32_t p = 0; p < P; ++p) E.put(ZERO, P + p, 0);
                break;
            case I_SEED: {
                uint32_t fl;
                const uint32_t tr = target(a.k, &fl);
                if (tr != kNone) E.put(ACC, tr, 0, kOne, kOne, (fl & kUFirst) ? kZeroC : tr);   // 1 * 1, gate open
                break;
            }
            case I_CKLD: {
                const uint32_t s = B.livein[a.k][a.j];
                uint32_t row = ckrow_base[a.k];
                for (uint32_t i = 0; i < a.j; ++i) row += I.nel[B.livein[a.k][i]];
                const uint32_t dst = rev_operand(s, a.k);
                for (uint32_t e = 0; e < I.nel[s]; e += kMaxCk)
                    E.put(CKLD, dst + e, 0, ck_row(row + e, std::min(kMaxCk, I.nel[s] - e)));
                Sch.ckpt_elems_loaded += I.nel[s];
                break;
            }
            case I_FWD: {
                auto opnd = [&](uint32_t s) { return rev_operand(s, a.j); };
                for (uint32_t b = 0; b < a.nops(); ++b) emit_fwd(a.op(b), opnd, opnd(a.op(b)));
                Sch.n_recompute_ops += a.nops();
                break;
            }
            case I_REV:
                for (uint32_t b = 0; b < a.nops(); ++b) emit_rev(a.op(b), a.j);
                break;
            case I_STG:
                E.put(STGRAD, P + a.k, 0, a.k);
                break;
            case I_ZERO: {   // +0 before the arm that would make the first contribution
                uint32_t fl;
                const uint32_t tr = target(a.k, &fl);
                for (uint32_t i = 0; i < I.nel[a.k]; ++i) E.put(ZERO, tr + i, 0);
                break;
            }
            case I_SKIP: {
                const auto &g = I.groups[a.k];
                const uint32_t pt = E.tmp();
                E.put(CMPLT, pt, 0, rev_operand(g.a, a.j), rev_operand(g.b, a.j));
                E.ops.push_back({kMarkBegin, 0, a.nb, {0, pt, 0, 0}});
                break;
            }
            case I_SKIPEND:
                E.ops.push_back({kMarkEnd, 0, 0, {0, 0, 0, 0}});
                break;
            default:
                break;
            }
        }
        Sch.n_regs = std::max(Sch.n_regs, E.tmp0 + E.used_tmp);
        Sch.n_temps_used = std::max(Sch.n_temps_used, E.used_tmp);
    }

    if (!full) return Sch;

    // ---- pack and encode: forward and reverse phases separately (the
    // reverse phase starts after every forward store)
    const uint32_t trash_row = Sch.n_ckpt_rows;   // kMaxBlock trash rows follow the checkpoints
    const uint32_t reg_bytes = 8 * (64 / S);      // byte offset of register r: r * reg_bytes
    std::vector<std::vector<UOp>> phases;
    if (with_grad) {
        phases.push_back(std::move(fwd_ops));
        phases.push_back(std::move(E.ops));
    } else {
        phases.push_back(std::move(E.ops));
    }
    std::vector<UOp> flat;
    std::vector<std::pair<uint32_t, uint32_t>> spans;   // (first op, count) per instruction
    for (auto &ph : phases) {
        // blocks between arm marks are packed apart; each arm is preceded by
        // a SKIP instruction that reads the predicate and jumps over the
        // arm's instructions when every lane of the wave decides the other way
        size_t b0 = 0;
        std::vector<UOp> block;
        UOp skip{};
        bool in_arm = false;
        auto flush = [&](size_t end) {
            block.assign(ph.begin() + b0, ph.begin() + end);
            const auto groups = pack(block, S);
            if (in_arm) {
                if (groups.size() > kSkipCountMask) throw std::length_error("skippable arm beyond the immediate field");
                skip.imm = uint32_t(groups.size()) | uint32_t(skip.flags) << kSkipSideShift;
                skip.flags = 0;
                spans.push_back({uint32_t(flat.size()), 1});
                flat.push_back(skip);
            }
            for (const auto &gq : groups) {
                spans.push_back({uint32_t(flat.size()), uint32_t(gq.size())});
                for (uint32_t j : gq) flat.push_back(block[j]);
            }
            Sch.n_uops += block.size();
        };
        for (size_t i = 0; i < ph.size(); ++i) {
            if (ph[i].form != kMarkBegin && ph[i].form != kMarkEnd) continue;
            flush(i);
            in_arm = ph[i].form == kMarkBegin;
            if (in_arm) {
                skip = UOp{SKIP, ph[i].imm, 0, {0, ph[i].f[1], 0, 0}};
                Sch.n_skips++;
            }
            b0 = i + 1;
        }
        flush(ph.size());
    }
    const uint32_t n_real = uint32_t(spans.size());
    // a skipped span ends before the END and holds no other skip test (the
    // device skips by counting instructions and never looks for END there)
    for (uint32_t i = 0, open_end = 0; i < n_real; ++i) {
        const UOp &u = flat[spans[i].first];
        if (u.form != SKIP) continue;
        const uint32_t n = u.imm & kSkipCountMask;
        if (i < open_end || uint64_t(i) + n >= n_real) throw std::logic_error("skipped span out of place");
        open_end = i + n + 1;
    }
    Sch.n_instr = n_real + 1;   // through the END
    const uint32_t n_chunks = n_real / kChunk + 1 + kFetchAhead;
    const uint32_t n_groups = n_real / kHeaderGroup + 1 + kFetchAhead;
    const size_t hdr_off = size_t(n_chunks) * kChunkWords;
    Sch.code.assign(hdr_off + size_t(n_groups) * kHeaderGroup, END);
    Sch.hdr_off = uint32_t(hdr_off);
    auto field = [&](uint64_t v) -> uint32_t {
        if (v > 0xFFFFFFFFull) throw std::length_error("register or index beyond the 32-bit fields of the device program");
        return uint32_t(v);
    };
    for (uint32_t i = 0; i < n_chunks * kChunk; ++i) {
        uint32_t *row0 = &Sch.code[size_t(i / kChunk) * kChunkWords + (i % kChunk) * 4];
        if (i >= n_real) {
            for (uint32_t r = 0; r < kRows; ++r) row0[r * kChunk * 4] = field(uint64_t(kSink) * reg_bytes);
            continue;
        }
        const auto [first, cnt] = spans[i];
        const UOp &u0 = flat[first];
        const uint32_t f = u0.form;
        uint32_t hdr = form_bits(f) | u0.imm << kImmShift;
        if (f == STLOSS || f == STGRAD) hdr = f | cnt << kImmShift;
        if (is_ckmove(f)) {   // the largest row count of the instruction's slots
            uint32_t mx = 1;
            for (uint32_t sl = 0; sl < cnt; ++sl) mx = std::max(mx, (flat[first + sl].f[1] >> kCkRowBits) + 1);
            hdr = f | mx << kImmShift;
        }
        for (uint32_t sl = 0; sl < S; ++sl) {
            UOp u = sl < cnt ? flat[first + sl] : u0;
            if (sl >= cnt) {
                if (writes_a(f)) u.f[0] = kSink;
                if (is_ckmove(f)) u.f[0] = kSink, u.f[1] = ck_row(trash_row, 1);
                u.flags = 0;
            }
            hdr |= (u.flags & kUFirst ? 1u : 0u) << (kFirstShift + sl);
            const uint32_t w[4] = {field(uint64_t(u.f[0]) * reg_bytes),
                                   x_is_index(f) ? u.f[1] : field(uint64_t(u.f[1]) * reg_bytes),
                                   field(uint64_t(u.f[2]) * reg_bytes), field(uint64_t(u.f[3]) * reg_bytes)};
            for (uint32_t r = sl * kRows / S; r < (sl + 1) * kRows / S; ++r)
                std::memcpy(row0 + r * kChunk * 4, w, 16);
        }
        Sch.code[hdr_off + i] = hdr;
        Sch.n_slots_used += cnt;
        Sch.n_mac += f == MAC;
        Sch.n_acc += f == ACC;
        Sch.n_msub += f == MSUB;
        Sch.n_block += f == DOTB || f == DOTBACC;
    }
    Sch.n_chunks = n_chunks;
    return Sch;
}

// Build with kTemps temporaries reserved; a program that uses none is built
// again with their registers given to the value pool (a wider spread of
// values means fewer reuses of one register, which would order otherwise
// independent micro-ops).  Deterministic: the lowering does not depend on
// the reservation.
Schedule build_fit(const Info &I, Builder &B, bool with_grad, uint32_t S, uint32_t reg_budget, bool full) {
    Schedule s = build(I, B, with_grad, S, reg_budget, kTemps, false);
    const uint32_t temps = s.n_temps_used ? kTemps : 0;
    if (temps == kTemps && !full) return s;
    return build(I, B, with_grad, S, reg_budget, temps, full);
}

Schedule forward_fit(const Tape &t, uint32_t slots, uint32_t reg_budget, uint32_t arm_min, uint32_t merge) {
    Info I(t);
    I.analyse();
    if (arm_min) I.find_arms(arm_min, merge);
    Builder B(I);
    B.set_cuts({0});
    B.resident.assign(I.N, 0);
    B.res_off.assign(I.N, 0);
    return build_fit(I, B, false, slots, reg_budget, true);
}

Schedule grad_fit(const Tape &t, uint32_t reg_budget, uint32_t slots, bool save_reads, uint32_t arm_min,
                  uint32_t merge) {
    Info I(t);
    I.analyse();
    if (arm_min) I.find_arms(arm_min, merge);
    uint64_t total = 0;
    for (uint32_t k = 0; k < I.N; ++k)
        if (I.kind[k] == K_COMP && I.vlive[k]) total += I.nel[k];
    const uint32_t kResidentAfter = 2;   // checkpointed in more segments -> keep resident
    // the search sizes registers only; the chosen size is built in full
    auto trial = [&](uint64_t S, bool full = false) {
        Builder B(I);
        B.save_reads = save_reads;
        B.resident.assign(I.N, 0);
        B.res_off.assign(I.N, 0);
        B.set_cuts(B.choose_cuts(S));
        B.plan(false);
        B.choose_residents(kResidentAfter);
        B.set_cuts(B.choose_cuts(S));
        B.plan(true);
        return build_fit(I, B, true, slots, reg_budget, full);
    };
    // Largest segment size (in value elements) whose register file fits the
    // budget: halve until it fits, then bisect between the fitting size and
    // the one above it.  If nothing fits, keep the smallest register file.
    uint64_t hi = std::max<uint64_t>(total, 1);
    Schedule best = trial(hi);
    uint64_t best_size = hi;
    if (best.n_regs <= reg_budget) return trial(best_size, true);
    uint64_t lo = hi;
    bool found = false;
    while (lo > 4) {
        lo /= 2;
        Schedule c = trial(lo);
        if (c.n_regs <= reg_budget) {
            best = std::move(c);
            best_size = lo;
            found = true;
            break;
        }
        if (c.n_regs < best.n_regs) {
            best = std::move(c);
            best_size = lo;
        }
        hi = lo;
    }
    if (!found) return trial(best_size, true);
    // invariant: lo fits, hi does not
    while (hi - lo > std::max<uint64_t>(8, lo / 16)) {
        uint64_t mid = lo + (hi - lo) / 2;
        Schedule c = trial(mid);
        if (c.n_regs <= reg_budget) {
            best = std::move(c);
            best_size = mid;
            lo = mid;
        } else {
            hi = mid;
        }
    }
    // A size that divides the trace evenly into as many segments cuts every
    // step of a loop at the same point (the largest fitting size drifts
    // through the steps): of the two, keep the schedule with fewer
    // instructions (Lotka-Volterra: 61,020 against 63,523).
    Schedule full = trial(best_size, true);
    const uint64_t even = total / std::max<uint32_t>(1, full.n_segments);
    if (even > 0 && even != best_size) {
        Schedule alt = trial(even, true);
        if (alt.n_regs <= reg_budget && alt.n_instr < full.n_instr) return alt;
    }
    return full;
}

}  // namespace

// Arms behind skip tests are an option of the layout, never a reason to
// exceed the register budget (or, where nothing fits it, the register file
// of the program without arms): with fewer branches per skip test (each
// merge keeps values live longer and forbids checkpoint cuts across it), and
// at last with no arms, until the register file fits.
namespace {
template <class F>
Schedule with_arms(uint32_t arm_min, uint32_t reg_budget, F fit) {
    Schedule plain = fit(0u, 1u);
    if (!arm_min) return plain;
    const uint32_t limit = std::max(reg_budget, plain.n_regs);
    for (uint32_t merge : {4u, 2u, 1u}) {
        Schedule s = fit(arm_min, merge);
        if (s.n_regs <= limit) return s;
    }
    return plain;
}
}  // namespace

Schedule schedule_forward(const Tape &t, uint32_t slots, uint32_t reg_budget, uint32_t arm_min) {
    return with_arms(arm_min, reg_budget,
                     [&](uint32_t a, uint32_t m) { return forward_fit(t, slots, reg_budget, a, m); });
}

Schedule schedule_grad(const Tape &t, uint32_t reg_budget, uint32_t slots, bool save_reads, uint32_t arm_min) {
    return with_arms(arm_min, reg_budget,
                     [&](uint32_t a, uint32_t m) { return grad_fit(t, reg_budget, slots, save_reads, a, m); });
}

}  // namespace ndvm
