// Host emulator of slot programs -- a checking tool for the scheduler, built
// into its own library (libndvm_emu.so) that only the CPU tests load; the
// product binding never calls it.
//
// It schedules a tape exactly as ndvm_tape_upload / ndvm_grad do and runs the
// resulting program lane by lane through the same micro-op handlers the GPU
// kernel uses.  Every slot of an instruction reads before any slot writes
// (writes are buffered until the instruction ends, as on the GPU); every
// register access is bounds-checked, every read of a never-written register
// is reported, and so is a slot that reads or writes a register another slot
// of the same instruction writes.  That exposes register-allocation,
// checkpoint, packing and first-contribution mistakes without a GPU.
#include <cmath>
#include <algorithm>
#include <cstdio>
#include <vector>

#include "common.h"
#include "sched.h"
#include "slot_exec.h"

using namespace ndvm;

namespace {

// Payload of one slot: register fields decoded from byte offsets into
// register numbers (the host context's handles).
struct P4 {
    uint32_t w[4], hdr, slot, reg_bytes;
    uint32_t *n_loaded;   // calls of loaded() (a hot handler makes exactly one)
    uint32_t a() const { return w[0] / reg_bytes; }
    uint32_t x() const { return w[1] / reg_bytes; }
    uint32_t y() const { return w[2] / reg_bytes; }
    uint32_t z() const { return w[3] / reg_bytes; }
    uint32_t ix() const { return w[1]; }
    uint32_t imm() const { return hdr >> slot::kImmShift; }
    bool first() const { return (hdr >> (slot::kFirstShift + slot)) & 1u; }
    void loaded() const { ++*n_loaded; }
};

struct HostCtx {
    double *regs;
    uint8_t *written;
    uint32_t n_regs, sink;
    const double *consts, *obs, *params;
    uint32_t n_consts, n_obs, n_params;
    double *loss, *grad;
    double *ckpt;
    uint32_t n_ckpt;   // rows including the trash row
    int *fault;        // first problem seen: 1 register range, 2 unwritten read, 3 pool/param/obs index,
                       // 4 ckpt row, 6 read of a register another slot writes, 7 two slots write one register,
                       // 8 form differs between slots, 9 output store or skip test inside a skipped arm,
                       // 10 a hot handler marked its operand reads other than once
    uint32_t cur_slot = 0;
    bool cur_dummy = false;   // an unused slot (result to the sink): its reads are never checked
    std::vector<std::pair<uint32_t, double>> *pending;
    std::vector<uint32_t> *pend_slot;

    static uint32_t uni(uint32_t x) { return x; }
    uint32_t slot() const { return cur_slot; }
    uint32_t *fault_reg = nullptr;   // register of the first fault (when it concerns one)
    void flag(int code, uint32_t r = 0xFFFFFFFFu) const {
        if (*fault == 0) {
            *fault = code;
            if (fault_reg) *fault_reg = r;
        }
    }
    void check_pending_read(uint32_t r) const {
        if (cur_dummy) return;
        for (size_t i = 0; i < pending->size(); ++i)
            if ((*pending)[i].first == r && (*pend_slot)[i] != cur_slot) flag(6);
    }
    static uint32_t adv(uint32_t h, uint32_t n) { return h + n; }
    double ld(uint32_t r) const {
        if (r >= n_regs) { flag(1); return NAN; }
        check_pending_read(r);
        if (!written[r] && !cur_dummy) flag(2, r);   // an unused slot may read an unwritten sink
        return regs[r];
    }
    double ld_raw(uint32_t r) const {
        if (r >= n_regs) { flag(1); return NAN; }
        if (r < sink || r >= sink + slot::kMaxBlock) check_pending_read(r);
        return regs[r];
    }
    void st(uint32_t r, double v) const {
        if (r >= n_regs) { flag(1); return; }
        if (poison) {
            if (cur_accum) return;
            v = NAN;
        }
        if (r < sink || r >= sink + slot::kMaxBlock)
            for (size_t i = 0; i < pending->size(); ++i)
                if ((*pending)[i].first == r && (*pend_slot)[i] != cur_slot) flag(7);
        pending->push_back({r, v});
        pend_slot->push_back(cur_slot);
    }
    void commit() const {
        for (const auto &pw : *pending) {
            regs[pw.first] = pw.second;
            written[pw.first] = 1;
        }
        pending->clear();
        pend_slot->clear();
    }
    double konst(uint32_t i) const {
        if (i >= n_consts) { flag(3); return NAN; }
        return consts[i];
    }
    double obsv(uint32_t i) const {
        if (i >= n_obs) { flag(3); return NAN; }
        return obs[i];
    }
    double param(uint32_t p) const {
        if (p >= n_params) { flag(3); return NAN; }
        return params[p];
    }
    void store_loss(double v, bool on) const {
        if (poison) flag(9);
        if (on) *loss = v;
    }
    void store_grad(uint32_t p, double v, bool on) const {
        if (poison) flag(9);
        if (!on) return;
        if (p >= n_params) { flag(3); return; }
        grad[p] = v;
    }
    void ckst(uint32_t row, double v) const {
        if (row >= n_ckpt) { flag(4); return; }
        ckpt[row] = poison ? NAN : v;
    }
    static void settle(double) {}
    void check_written(uint32_t r) const {
        if (r < n_regs && !written[r] && !cur_dummy) flag(2, r);
    }
    // SKIP, one lane at a time: the lane skips the arm it does not take (the
    // most skipping any wave of lanes could do)
    mutable uint32_t skip = 0;
    bool never_skip = false;
    // An instruction of an arm this lane skips.  On the GPU its registers
    // keep whatever they held; here every value it would form anew (forward
    // values, temporaries, first contributions) is set to NaN and every
    // adjoint it would add to keeps its value, so a result that depends on a
    // skipped arm comes out NaN or differs from the run without skipping.
    bool poison = false;
    bool cur_accum = false;   // the slot's writes add to their own register (not formed anew)
    void skip_arm(bool then_taken, uint32_t imm) const {
        const bool else_arm = (imm >> slot::kSkipSideShift) & 1u;
        if (poison) flag(9);
        if (!never_skip && (else_arm ? then_taken : !then_taken)) skip = imm & slot::kSkipCountMask;
    }
    double ckld(uint32_t row) const {
        if (row >= n_ckpt) { flag(4); return NAN; }
        return ckpt[row];
    }
};

// forms whose writes add to the register written (an adjoint update that is
// not the first contribution)
bool accumulates(uint32_t form, const P4 &p) {
    switch (form) {
    case slot::ACC: return p.z() == p.a();
    case slot::MACG: case slot::ACCD: case slot::ACCND: case slot::DOTACC: case slot::ACCSEL: case slot::ACCABS:
    case slot::DOTBACC:
        return !p.first();
    default:
        return false;
    }
}

// with_grad: 0 forward only, 1 gradient (recompute policy), 2 gradient (save
// policy); arm_min: smallest arm behind a skip test (0: none)
Schedule schedule(const Tape &t, int with_grad, uint32_t reg_budget, uint32_t slots, uint32_t arm_min) {
    return with_grad ? schedule_grad(t, reg_budget, slots, with_grad == 2, arm_min)
                     : schedule_forward(t, slots, reg_budget, arm_min);
}
// mode bits 8 / 16: arms as the NDVM_BRANCH_SKIP option lays them out / every
// arm however small
uint32_t arm_min_of(int mode) { return (mode & 16) ? 1 : (mode & 8) ? kArmMinElems : 0; }

}  // namespace

extern "C" {

/*
 * Schedule `tape` (forward-only when with_grad == 0, else the gradient
 * program for `reg_budget` registers) with `slots` micro-ops per instruction
 * and run it for L lanes on the host.  with_grad: 0 forward only, 1 gradient
 * (recompute policy), 2 gradient (save policy); + 4: never skip a branch arm;
 * + 8: branch arms behind skip tests (as the NDVM_BRANCH_SKIP option lays
 * them out); + 16: every branch arm behind a skip test, however small.
 * stats (optional, 11 entries): n_regs, n_ckpt_rows, n_segments, n_instr, fwd
 * ops, recompute ops, reverse ops, checkpoint elements stored, micro-ops,
 * slots used, skippable arms.
 * Returns 0, an ndvm_status from parsing, or 100 + fault code.
 */
int ndvm_emu_run(const uint8_t *tape, size_t len, int with_grad, uint32_t reg_budget, uint32_t slots,
                 const double *params, int64_t L, int64_t ld_p, const double *obs, int64_t n_obs, double *loss,
                 double *grad, int64_t ld_g, uint64_t *stats) {
    const bool never_skip = (with_grad & 4) != 0;   // run both arms of every branch
    const uint32_t arm_min = arm_min_of(with_grad);
    with_grad &= 3;
    Tape t;
    ndvm_status st = parse_tape(tape, len, &t);
    if (st != NDVM_OK) return st;
    if (n_obs != int64_t(t.n_obs)) return NDVM_E_ARG;
    if (slots != 1 && slots != 2 && slots != 4) return NDVM_E_ARG;
    Schedule S;
    try {
        S = schedule(t, with_grad, reg_budget, slots, arm_min);
    } catch (const std::exception &e) {
        set_error(e.what());
        return NDVM_E_UNSUPPORTED;
    }
    if (stats) {
        uint64_t v[11] = {S.n_regs, S.n_ckpt_rows, S.n_segments, S.n_instr, S.n_fwd_ops,
                          S.n_recompute_ops, S.n_rev_ops, S.ckpt_elems_stored, S.n_uops, S.n_slots_used,
                          S.n_skips};
        for (int i = 0; i < 11; ++i) stats[i] = v[i];
    }
    const uint32_t sink = 2 * t.n_params;
    std::vector<double> regs(S.n_regs), ck(size_t(S.n_ckpt_rows) + slot::kMaxBlock);
    std::vector<uint8_t> written(S.n_regs);
    std::vector<std::pair<uint32_t, double>> pending;
    std::vector<uint32_t> pend_slot;
    const uint32_t K = slot::kChunk;
    const uint32_t reg_bytes = 8 * (64 / slots);
    for (int64_t l = 0; l < L; ++l) {
        std::fill(written.begin(), written.end(), 0);
        int fault = 0;
        HostCtx c{regs.data(), written.data(), S.n_regs, sink, S.consts.data(), obs, params + l * ld_p,
                  uint32_t(S.consts.size()), uint32_t(n_obs), t.n_params, loss + l,
                  grad ? grad + l * ld_g : nullptr, ck.data(), S.n_ckpt_rows + slot::kMaxBlock, &fault, 0, false, &pending,
                  &pend_slot};
        uint32_t fault_reg = 0xFFFFFFFFu, fault_form = 0;
        uint64_t fault_instr = 0;
        c.fault_reg = &fault_reg;
        c.never_skip = never_skip;
        bool ended = false;
        uint32_t skipped = 0;   // instructions of a skipped arm still to come
        for (uint64_t i = 0; i < uint64_t(S.n_chunks) * K && !ended && !fault; ++i) {
            c.poison = skipped > 0;
            if (skipped) --skipped;
            const uint32_t hdr = S.code[S.hdr_off + i];
            const uint32_t form = hdr & slot::kFormMask;
            fault_instr = i;
            fault_form = form;
            if (form == slot::END) {
                ended = true;
                break;
            }
            for (uint32_t sl = 0; sl < slots; ++sl) {
                // slot sl's words sit in rows sl * 4 / S ..; take the first
                const uint32_t r = sl * slot::kRows / slots;
                const uint32_t *w = &S.code[size_t(i / K) * slot::kChunkWords + (size_t(r) * K + i % K) * 4];
                uint32_t n_loaded = 0;
                const P4 p{{w[0], w[1], w[2], w[3]}, hdr, sl, reg_bytes, &n_loaded};
                c.cur_slot = sl;
                c.cur_dummy = c.poison || (slot::writes_a(form) && p.a() == sink) ||
                              (form == slot::CKST && (p.ix() & slot::kCkRowMask) == S.n_ckpt_rows);
                c.cur_accum = accumulates(form, p);
                if (slot::is_hot(form)) {
                    slotx::exec_hot(c, form, p);
                    if (n_loaded != 1) c.flag(10);
                } else
                    slotx::exec_cold(c, form, p);
            }
            c.commit();
            if (c.skip) {   // the arm's instructions run poisoned
                skipped = c.skip;
                c.skip = 0;
            }
        }
        if (!ended && !fault) fault = 5;
        if (fault) {
            char m[160];
            std::snprintf(m, sizeof m, "emulator fault %d in lane %lld at instruction %llu (form %u), register %u",
                          fault, (long long)l, (unsigned long long)fault_instr, fault_form, fault_reg);
            set_error(m);
            return 100 + fault;
        }
    }
    return 0;
}

/*
 * Copy the device program the scheduler makes for `tape` (slot words,
 * chunk-major ([chunk][row][instr][4]), then the headers; slot.h) into `out`
 * when it holds `cap` words;
 * returns the number of words, or -1 on an error.
 */
int64_t ndvm_emu_program(const uint8_t *tape, size_t len, int with_grad, uint32_t reg_budget, uint32_t slots,
                         uint32_t *out, size_t cap, uint32_t *hdr_off) {
    Tape t;
    if (parse_tape(tape, len, &t) != NDVM_OK) return -1;
    Schedule S;
    try {
        S = schedule(t, with_grad & 3, reg_budget, slots, arm_min_of(with_grad));
    } catch (const std::exception &e) {
        set_error(e.what());
        return -1;
    }
    const size_t n = S.code.size();
    if (out && cap >= n) std::copy(S.code.begin(), S.code.end(), out);
    if (hdr_off) *hdr_off = S.hdr_off;
    return int64_t(n);
}

const char *ndvm_emu_error(void) { return get_error(); }

}  // extern "C"
