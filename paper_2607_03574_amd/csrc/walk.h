// Device walker: definitions shared by its host part (walk_host.cpp) and its
// kernel (walk.hip).
//
// The walker runs the structural walk of a stack-bytecode program on the
// GPU -- the device interpreter the paper leaves as designed but unbuilt
// (Section 9, "What remains designed and unbuilt"; Appendix A): one wave
// walks the program for 64 lanes.  Structure (program counter, operand stack, locals,
// loop counters) is the same for every lane and is kept once per wave; each
// numeric word records one node whose per-lane value goes to the wave's
// value rows in HBM (define-by-run, Section 3.4).  A numeric IFLT runs each
// arm under the mask of the lanes that take it (one ballot; an arm no lane
// takes is skipped), and at ENDIF every stack position and local the two
// arms left different becomes a MERGE node that picks, per lane, the value
// of the arm the lane took (Section 6, lane-masked divergent control).  The
// reverse sweep walks the recorded nodes backwards with per-lane adjoints
// (Appendix C, table tab:adjoints).
#pragma once
#include <cstdint>

namespace ndvm {
namespace walk {

// One program in the device buffer.  Offsets count 32-bit words from the
// start of the buffer; the constants start 8-byte aligned.
struct ProgDesc {
    uint32_t code_off;    // n_instr instruction words, 2 x u32 each: op | a << 8 | pops << 16 | pushes << 18, imm
    uint32_t match_off;   // n_instr int32: LOOP -> ENDLOOP, IFLT -> ELSE, ELSE -> ENDIF, else -1
    uint32_t const_off;   // n_consts doubles
    uint32_t n_instr;
    uint32_t n_params, n_obs;
    uint32_t n_nodes;     // bound on the nodes one wave records (parameters included)
    uint32_t depth;       // bound on the operand stack depth
    uint32_t n_locals;    // locals referenced (largest index + 1)
    uint32_t n_frames;    // bound on IFLT nesting
    uint32_t n_loops;     // bound on LOOP nesting
    uint32_t n_steps;     // bound on the words one walk executes (the walk stops there)
};

// A node number with this bit set on the operand stack, in a local or as a
// recorded operand is a constant or observation: it takes no adjoint.
constexpr uint32_t kLeafBit = 0x80000000u;

// Node kinds beyond the bytecode's numeric opcodes (which keep their numbers).
constexpr uint32_t kLeaf = 0x01;    // constant or observation: takes no adjoint
constexpr uint32_t kParam = 0x02;   // parameter p = node p
constexpr uint32_t kMerge = 0x40;   // per-lane pick of two arms' values (a if the lane took the first arm)

// Recorded node (one per node and wave, 16 bytes): its kind and operand
// nodes; for a MERGE, `mask` indexes the ballot word of the lanes that took
// the first arm (stored after the node records).
struct Node {
    uint32_t op, a, b, mask;
};

// Per-wave workspace: values[n_nodes][64], adjoints[n_nodes][64] (fp64),
// nodes[n_nodes], ballot words[n_nodes] (u64, MERGE nodes only).
constexpr uint64_t ws_bytes_per_node() { return 64 * 8 * 2 + sizeof(Node) + 8; }

// LDS of one wave.  Rows of 64 doubles first: the parameters' values, then
// the operand stack's and the locals' values during the forward walk, whose
// rows the parameters' adjoints take over in the reverse sweep.  Then 32-bit
// words: the operand stack's and locals' node numbers, loop frames (start,
// trips, counter), IFLT frames (masks, phase, two snapshots of stack +
// locals node numbers), and one flag bit per node (adjoint row written).
constexpr uint32_t kFrameFixed = 8;
constexpr uint32_t lds_rows(uint32_t depth, uint32_t n_locals, uint32_t n_params) {
    const uint32_t fwd = depth + n_locals;
    return n_params + (fwd > n_params ? fwd : n_params);
}
constexpr uint32_t lds_words(uint32_t depth, uint32_t n_locals, uint32_t n_loops, uint32_t n_frames,
                          uint32_t n_nodes) {
    const uint32_t snap = depth + n_locals;
    return depth + n_locals + 3 * n_loops + n_frames * (kFrameFixed + 2 * snap) + (n_nodes + 31) / 32;
}
constexpr uint64_t lds_bytes(uint32_t depth, uint32_t n_locals, uint32_t n_loops, uint32_t n_frames, uint32_t n_nodes,
                          uint32_t n_params) {
    return 512ull * lds_rows(depth, n_locals, n_params) + 4ull * lds_words(depth, n_locals, n_loops, n_frames, n_nodes);
}

// Limits the host validator enforces.
constexpr uint32_t kMaxDepth = 64, kMaxLocals = 32, kMaxFrames = 32, kMaxLoops = 32;
constexpr uint64_t kMaxLdsBytes = 64 * 1024;   // a workgroup's LDS
constexpr uint64_t kMaxNodes = 1u << 22;   // node * 64 + lane fits 32 bits

struct Args {
    const uint32_t *buf;        // device buffer: ProgDesc[n_prog] then code, matches, constants
    uint32_t n_prog;
    int64_t L;                  // lanes per program
    const double *params;       // [n_prog][L][ld_p] (program stride prog_stride_p)
    int64_t ld_p, prog_stride_p;
    const double *obs;          // shared by every program
    double *loss;               // [n_prog][L]
    double *grad;               // [n_prog][L][ld_g] (program stride prog_stride_g)
    int64_t ld_g, prog_stride_g;
    uint8_t *ws;                // per wave slot: n_nodes_max * ws_bytes_per_node() bytes
    uint32_t n_nodes_max;       // nodes per wave slot
    uint32_t lds_bytes;         // LDS bytes per wave
    uint32_t depth, n_locals, n_loops, n_frames, n_params;   // LDS layout bounds (maxima over the programs)
    uint64_t n_items;           // work items: n_prog * ceil(L / 64)
    int *status;                // device word: 0, or a nonzero code when a wave met a bound it must not pass
};

}  // namespace walk
}  // namespace ndvm
