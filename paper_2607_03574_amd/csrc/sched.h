// Tape scheduler: validated tape -> device program for the replay kernel.
#pragma once
#include <cstdint>
#include <vector>

#include "common.h"

namespace ndvm {

struct Schedule {
    std::vector<uint32_t> code;   // slot words, chunk-major ([chunk][row][instr][4]), then headers (slot.h)
    std::vector<double> consts;   // constant pool: the tape's, then 1, -1, -0, 2, 1e-8, +0
    uint32_t slots = 1;           // micro-ops per instruction (threads per lane)
    uint32_t n_regs = 0;          // lane registers used
    uint32_t n_ckpt_rows = 0;     // checkpoint rows (fp64 per lane); slot::kMaxBlock trash rows follow
    uint32_t n_segments = 1;
    uint32_t n_chunks = 0;        // fetch chunks of the program, read-ahead chunks included
    uint32_t hdr_off = 0;         // word offset of the headers in code
    uint32_t static_regs = 0, fwd_regs = 0, rev_regs = 0;
    uint32_t n_temps_used = 0;    // temporaries the lowering used (0: their registers went to the value pool)
    uint64_t n_instr = 0, n_uops = 0, n_slots_used = 0;
    uint64_t n_fwd_ops = 0, n_recompute_ops = 0, n_rev_ops = 0;
    uint64_t ckpt_elems_stored = 0, ckpt_elems_loaded = 0;
    uint32_t n_skips = 0;         // skippable branch arms (SKIP instructions)
    uint64_t n_mac = 0, n_acc = 0, n_msub = 0, n_block = 0;   // instructions of the most frequent forms
};

// Smallest branch arm (in value elements) laid out behind a skip test: a
// smaller one costs more in its skip test and in the packing it breaks than
// a wave could save by skipping it.
constexpr uint32_t kArmMinElems = 8;

// Forward-only program (loss[L]) with `slots` micro-ops per instruction;
// values spread over up to `reg_budget` registers.  With arm_min > 0, the
// arms of numeric branches with at least arm_min value elements are laid out
// behind skip tests (a wave whose lanes all decide a branch one way skips the
// other arm).
Schedule schedule_forward(const Tape &t, uint32_t slots, uint32_t reg_budget, uint32_t arm_min = 0);

// Forward + reverse program (loss[L], grad[L, P]); cuts the tape into
// checkpoint segments so that the lane register file fits `reg_budget`
// registers when possible.  With save_reads, every value an adjoint rule
// reads is stored when the forward sweep computes it and restored for its
// segment's reverse sweep, so nothing is recomputed; otherwise only segment
// inputs are stored and each segment recomputes what its rules read.
// arm_min as for schedule_forward (both sweeps).
Schedule schedule_grad(const Tape &t, uint32_t reg_budget, uint32_t slots, bool save_reads = false,
                       uint32_t arm_min = 0);

}  // namespace ndvm
