// Host emulator of the device program -- a checking tool for the scheduler,
// built into its own library (libndvm_emu.so) that only the CPU tests load;
// the product binding never calls it.
//
// It schedules a tape exactly as ndvm_tape_upload / ndvm_grad do and runs the
// resulting program lane by lane through the same instruction handlers the
// GPU kernel uses, with every register access bounds-checked and every read
// of a never-written register reported.  That exposes register-allocation,
// checkpoint and first-contribution mistakes without a GPU.
#include <cmath>
#include <algorithm>
#include <cstdio>
#include <vector>

#include "common.h"
#include "replay.h"
#include "sched.h"

using namespace ndvm;

namespace {

struct HostCtx {
    const uint32_t *code_end;
    double *regs;
    uint8_t *written;
    uint32_t n_regs;
    const double *consts, *obs, *params;
    uint32_t n_consts, n_obs, n_params;
    double *loss, *grad;
    double *ckpt;
    uint32_t n_ckpt;
    int *fault;       // first problem seen: 1 register range, 2 unwritten read, 3 pool, 4 ckpt,
                      // 5 program fetch beyond the padded program

    static uint32_t uni(uint32_t x) { return x; }
    static bool all(bool b) { return b; }
    using Chunk = const uint32_t *;
    Chunk load_chunk(const uint32_t *p) const {
        if (p + isa::kChunkWords > code_end) flag(5);
        return p;
    }
    static const uint32_t *instr(Chunk ch, uint32_t i) { return ch + i * isa::kWords; }
    static uint32_t aux_word(const uint32_t *aux, uint32_t i) { return aux[i]; }
    void flag(int code) const {
        if (*fault == 0) *fault = code;
    }
    double ld(uint32_t r) const {
        if (r >= n_regs) { flag(1); return NAN; }
        if (!written[r]) flag(2);
        return regs[r];
    }
    double ld_raw(uint32_t r) const {
        if (r >= n_regs) { flag(1); return NAN; }
        return regs[r];
    }
    static uint32_t half(uint32_t word, int hi) { return hi ? word >> 16 : word & 0xFFFFu; }
    double ldh(uint32_t word, int hi) const { return ld(half(word, hi)); }
    double ldh_raw(uint32_t word, int hi) const { return ld_raw(half(word, hi)); }
    void sth(uint32_t word, int hi, double v) const { st(half(word, hi), v); }
    void st(uint32_t r, double v) const {
        if (r >= n_regs) { flag(1); return; }
        regs[r] = v;
        written[r] = 1;
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
    void store_loss(double v) const { *loss = v; }
    void store_grad(uint32_t p, double v) const {
        if (p >= n_params) { flag(3); return; }
        grad[p] = v;
    }
    void ckpt_st(uint32_t row, double v) const {
        if (row >= n_ckpt) { flag(4); return; }
        ckpt[row] = v;
    }
    double ckpt_ld(uint32_t row) const {
        if (row >= n_ckpt) { flag(4); return NAN; }
        return ckpt[row];
    }
};

}  // namespace

extern "C" {

/*
 * Schedule `tape` (forward-only when with_grad == 0, else the gradient
 * program for `reg_budget` registers) and run it for L lanes on the host.
 * stats (optional, 8 entries): n_regs, n_ckpt_rows, n_segments, n_instr,
 * fwd ops, recompute ops, reverse ops, checkpoint elements stored.
 * Returns 0, an ndvm_status from parsing, or 100 + fault code.
 */
int ndvm_emu_run(const uint8_t *tape, size_t len, int with_grad, uint32_t reg_budget, const double *params,
                 int64_t L, int64_t ld_p, const double *obs, int64_t n_obs, double *loss, double *grad,
                 int64_t ld_g, uint64_t *stats) {
    Tape t;
    ndvm_status st = parse_tape(tape, len, &t);
    if (st != NDVM_OK) return st;
    if (n_obs != int64_t(t.n_obs)) return NDVM_E_ARG;
    Schedule S = with_grad ? schedule_grad(t, reg_budget) : schedule_forward(t);
    if (stats) {
        uint64_t v[8] = {S.n_regs, S.n_ckpt_rows, S.n_segments, S.n_instr, S.n_fwd_ops,
                         S.n_recompute_ops, S.n_rev_ops, S.ckpt_elems_stored};
        for (int i = 0; i < 8; ++i) stats[i] = v[i];
    }
    std::vector<double> regs(S.n_regs), ck(S.n_ckpt_rows);
    std::vector<uint8_t> written(S.n_regs);
    for (int64_t l = 0; l < L; ++l) {
        std::fill(written.begin(), written.end(), 0);
        int fault = 0;
        HostCtx c{S.code.data() + S.code.size(), regs.data(), written.data(), S.n_regs, S.consts.data(), obs, params + l * ld_p,
                  uint32_t(S.consts.size()), uint32_t(n_obs), t.n_params, loss + l,
                  grad ? grad + l * ld_g : nullptr, ck.data(), S.n_ckpt_rows, &fault};
        replay::run(c, S.code.data(), S.aux.data());
        if (fault) {
            char m[96];
            std::snprintf(m, sizeof m, "emulator fault %d in lane %lld", fault, (long long)l);
            set_error(m);
            return 100 + fault;
        }
    }
    return 0;
}

/*
 * Copy the device program the scheduler makes for `tape` (words, isa::kWords
 * per instruction, END-terminated) into `out` when it holds `cap` words;
 * returns the number of words, or -1 on a parse error.
 */
int64_t ndvm_emu_program(const uint8_t *tape, size_t len, int with_grad, uint32_t reg_budget, uint32_t *out,
                         size_t cap) {
    Tape t;
    if (parse_tape(tape, len, &t) != NDVM_OK) return -1;
    Schedule S = with_grad ? schedule_grad(t, reg_budget) : schedule_forward(t);
    const size_t n = size_t(S.n_instr) * isa::kWords;
    if (out && cap >= n) std::copy(S.code.begin(), S.code.begin() + n, out);
    return int64_t(n);
}

const char *ndvm_emu_error(void) { return get_error(); }

}  // extern "C"
