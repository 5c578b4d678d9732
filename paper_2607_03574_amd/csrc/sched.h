// Tape scheduler: validated tape -> device program for the replay kernel.
#pragma once
#include <cstdint>
#include <vector>

#include "common.h"

namespace ndvm {

struct Schedule {
    std::vector<uint32_t> code;   // instructions, isa::kWords words each
    std::vector<uint32_t> aux;    // operand / target lists
    std::vector<double> consts;   // constant pool: the tape's, then 1, -1, -0
    uint32_t n_regs = 0;          // lane registers used
    uint32_t n_ckpt_rows = 0;     // checkpoint rows (fp64 per lane)
    uint32_t n_segments = 1;
    uint32_t static_regs = 0, fwd_regs = 0, rev_regs = 0;
    uint64_t n_instr = 0, n_fwd_ops = 0, n_recompute_ops = 0, n_rev_ops = 0;
    uint64_t ckpt_elems_stored = 0, ckpt_elems_loaded = 0;
    uint64_t n_bundles = 0;       // instructions holding 2 or 3 ops
    uint64_t n_bundled_ops = 0;   // ops inside those
};

// Forward-only program (loss[L]).
Schedule schedule_forward(const Tape &t);

// Forward + reverse program (loss[L], grad[L, P]); cuts the tape into
// checkpoint segments so that the lane register file fits `reg_budget`
// registers when possible.
Schedule schedule_grad(const Tape &t, uint32_t reg_budget);

}  // namespace ndvm
