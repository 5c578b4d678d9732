// Replay kernel: forward replay and reverse sweep of a scheduled tape.  A wave
// of 64 threads serves 64/S lanes (parameter vectors) with S slots each
// (Section 3.5: one structural walk, numeric payloads widened over the batch
// axis; here the batch axis and the tape's own parallelism share the wave).
//
// Every instruction is wave-uniform in its form and immediates, so all
// threads follow the same control; per-lane numeric branches were turned into
// selects by the trace producer.  The program is fetched four instructions
// at a time, one dword per thread, and row broadcasts hand each thread its
// slot's micro-op fields; the thread finds its operands
// in the lane's register file in LDS (register r of lane l at
// lds[r * 64/S + l]) and writes one fp64 result.  Registers past the LDS
// budget live in lane-contiguous workspace rows.  Small matrices are spread
// over the slots element by element; nothing here is a dense contraction, so
// no matrix cores are used.
#include <hip/hip_runtime.h>

#include <mutex>

#include "slot.h"
#include "slot_exec.h"

namespace ndvm {
namespace {

#define AS_LDS __attribute__((address_space(3)))
#define AS_GLOBAL __attribute__((address_space(1)))

template <int S, bool kSpill>
struct DevCtx {
    static constexpr int LW = 64 / S;   // lanes per wave
    AS_GLOBAL double *spill;
    const AS_GLOBAL double *consts, *obs, *params;
    AS_GLOBAL double *loss, *grad, *ckpt;
    int64_t lane, lc, Lpad, ld_p, ld_g;
    uint32_t r_lds, lane_addr, stride, slot_;
    bool active;

    __device__ __forceinline__ static uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }
    __device__ __forceinline__ uint32_t slot() const { return slot_; }
    // LDS address of the register named by the low 24 bits of f: one
    // v_mad_u32_u24, whose 24-bit multiply ignores the field's high byte
    __device__ __forceinline__ AS_LDS double *rp(uint32_t f) const {
        uint32_t a;
        asm("v_mad_u32_u24 %0, %1, %2, %3" : "=v"(a) : "v"(f), "v"(stride), "v"(lane_addr));
        return (AS_LDS double *)(size_t)a;
    }
    __device__ __forceinline__ double ld(uint32_t f) const {
        if (!kSpill) return *rp(f);
        const uint32_t r = f & slot::kFieldMask;
        if (r < r_lds) return *rp(r);
        return spill[int64_t(r - r_lds) * Lpad + lane];
    }
    __device__ __forceinline__ double ld_raw(uint32_t f) const { return ld(f); }
    __device__ __forceinline__ void st(uint32_t f, double v) const {
        if (!kSpill) {
            *rp(f) = v;
            return;
        }
        const uint32_t r = f & slot::kFieldMask;
        if (r < r_lds)
            *rp(r) = v;
        else
            spill[int64_t(r - r_lds) * Lpad + lane] = v;
    }
    __device__ __forceinline__ double obsv(uint32_t i) const { return obs[i]; }
    __device__ __forceinline__ double konst(uint32_t i) const { return consts[i]; }
    __device__ __forceinline__ double param(uint32_t p) const { return params[lc * ld_p + p]; }
    __device__ __forceinline__ double ckld(uint32_t row) const { return ckpt[int64_t(row) * Lpad + lane]; }
    __device__ __forceinline__ void ckst(uint32_t row, double v) const { ckpt[int64_t(row) * Lpad + lane] = v; }
    __device__ __forceinline__ void store_loss(double v, bool on) const {
        if (on && active) loss[lane] = v;
    }
    __device__ __forceinline__ void store_grad(uint32_t p, double v, bool on) const {
        if (on && active) grad[lane * ld_g + p] = v;
    }
};

// Word j of this thread's row, broadcast to the whole row (DPP
// row_newbcast:j); the lane index is a compile-time constant.
template <int J>
__device__ __forceinline__ uint32_t row_word(uint32_t v) {
    return uint32_t(__builtin_amdgcn_mov_dpp(int(v), 0x150 + J, 0xF, 0xF, false));
}
__device__ __forceinline__ uint32_t lane_word(uint32_t v, int lane) {
    return uint32_t(__builtin_amdgcn_readlane(int(v), lane));
}

// Payload of instruction P of a chunk: this thread's words (row broadcasts);
// the uniform words that carry the immediates are read from the chunk only
// by the forms that use them.
template <int P>
struct ChunkPayload {
    uint32_t x, y, z, w;
    uint32_t ch;
    __device__ __forceinline__ uint32_t u1() const { return lane_word(ch, 4 * P + 1); }
    __device__ __forceinline__ uint32_t u2() const { return lane_word(ch, 4 * P + 2); }
    __device__ __forceinline__ uint32_t u3() const { return lane_word(ch, 4 * P + 3); }
};
// Payload of a cold instruction, immediates read out
struct Payload {
    uint32_t x, y, z, w;
    uint32_t v1, v2, v3;
    __device__ __forceinline__ uint32_t u1() const { return v1; }
    __device__ __forceinline__ uint32_t u2() const { return v2; }
    __device__ __forceinline__ uint32_t u3() const { return v3; }
};

// Cold micro-ops run out of line: their library code branches per lane, and
// keeping those branches out of the replay loop leaves its hot part free of
// divergent control flow.  Returns 1 for END.
template <class C>
__device__ __attribute__((noinline)) uint32_t cold_call(const C &c, uint32_t form, Payload p) {
    if (form == slot::END) return 1;
    slotx::exec_cold(c, form, p);
    return 0;
}

// Instruction P of the chunk held in `ch` (one dword per thread); returns 1
// when it is END.
template <int P, class C>
__device__ __forceinline__ uint32_t step(const C &c, uint32_t ch) {
    const uint32_t form = (lane_word(ch, 4 * P) >> slot::kFormShift) & 63u;
    const ChunkPayload<P> p{row_word<4 * P>(ch), row_word<4 * P + 1>(ch), row_word<4 * P + 2>(ch),
                            row_word<4 * P + 3>(ch), ch};
    if (form < slot::HOT_END) {
        slotx::exec_hot(c, form, p);
        return 0;
    }
    return cold_call(c, form, Payload{p.x, p.y, p.z, p.w, p.u1(), p.u2(), p.u3()});
}

// Execute a slot program until END: the four instructions of each chunk in
// straight-line code, chunk c + 2 requested when chunk c starts (two chunks
// of END follow the program's END for this read-ahead; instructions after
// END in its chunk are END too).
template <int S, bool kSpill>
__device__ __forceinline__ void run(const DevCtx<S, kSpill> &c, const uint32_t *prog) {
    static_assert(slot::kChunk == 4 && slot::kFetchAhead == 2, "the fetch below reads four-instruction chunks two ahead");
    const AS_GLOBAL uint32_t *pc = (const AS_GLOBAL uint32_t *)prog + threadIdx.x;
    constexpr uint32_t W = slot::kChunkWords;
    uint32_t cur = pc[0], n1 = pc[W];
    for (;;) {
        pc += W;
        const uint32_t n2 = pc[W];
        uint32_t ended = step<0>(c, cur);
        ended |= step<1>(c, cur);
        ended |= step<2>(c, cur);
        ended |= step<3>(c, cur);
        if (ended) return;
        cur = n1;
        n1 = n2;
    }
}

}  // namespace

template <int S, bool kSpill>
__device__ __forceinline__ void replay_body(const LaunchArgs &A, const ProgStatic *__restrict__ table,
                                            const ProgStatic &single) {
    extern __shared__ double lds_regs[];
    constexpr int LW = 64 / S;
    const uint32_t q = blockIdx.y;
    const ProgStatic D = table ? table[q] : single;
    DevCtx<S, kSpill> c;
    const int t = threadIdx.x, l = t % LW;
    c.slot_ = uint32_t(t / LW);
    c.lane = int64_t(blockIdx.x) * LW + l;
    c.active = c.lane < A.L;
    c.lc = c.active ? c.lane : A.L - 1;
    c.lane_addr = uint32_t(size_t((AS_LDS double *)lds_regs + l));
    c.stride = uint32_t(LW * sizeof(double));
    c.spill = (AS_GLOBAL double *)(A.ws + int64_t(D.spill_row0) * A.Lpad);
    c.ckpt = (AS_GLOBAL double *)(A.ws + int64_t(D.ckpt_row0) * A.Lpad);
    c.consts = (const AS_GLOBAL double *)D.consts;
    c.obs = (const AS_GLOBAL double *)A.obs;
    c.params = (const AS_GLOBAL double *)(A.params + int64_t(q) * A.prog_stride_p);
    c.loss = (AS_GLOBAL double *)(A.loss + int64_t(q) * A.L);
    c.grad = (AS_GLOBAL double *)(A.grad + int64_t(q) * A.prog_stride_g);
    c.Lpad = A.Lpad;
    c.ld_p = A.ld_p;
    c.ld_g = A.ld_g;
    c.r_lds = D.r_lds;
    run(c, D.prog);
}

// All lane registers in LDS (the usual case: the scheduler fits the register
// file to the launch's LDS budget).
template <int S>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4)))
ndvm_replay(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    replay_body<S, false>(A, table, single);
}

// Registers beyond r_lds spill to lane-contiguous workspace rows.
template <int S>
__global__ void __launch_bounds__(64)
ndvm_replay_spill(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    replay_body<S, true>(A, table, single);
}

// Many programs in one launch, only some of which spill: each workgroup takes
// the variant its program needs, so one spilling program does not slow the
// others down.
template <int S>
__global__ void __launch_bounds__(64)
ndvm_replay_per_program(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    if (table[blockIdx.y].spills)
        replay_body<S, true>(A, table, single);
    else
        replay_body<S, false>(A, table, single);
}

namespace {

template <int S>
hipError_t launch_s(const LaunchArgs &A, const ProgStatic *d_table, const ProgStatic &single, uint32_t n_prog,
                    uint32_t r_lds, int variant, hipStream_t stream) {
    static std::once_flag once[64];
    int dev = 0;
    (void)hipGetDevice(&dev);
    std::call_once(once[dev & 63], [dev]() {
        int max_smem = 0;
        (void)hipDeviceGetAttribute(&max_smem, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&ndvm_replay<S>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&ndvm_replay_spill<S>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&ndvm_replay_per_program<S>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
    });
    constexpr int LW = 64 / S;
    dim3 grid(uint32_t((A.L + LW - 1) / LW), n_prog), block(64);
    size_t smem = size_t(r_lds) * LW * sizeof(double);
    if (variant == kPerProgram && d_table)
        hipLaunchKernelGGL(ndvm_replay_per_program<S>, grid, block, smem, stream, A, d_table, single);
    else if (variant == kSpill || variant == kPerProgram)
        hipLaunchKernelGGL(ndvm_replay_spill<S>, grid, block, smem, stream, A, d_table, single);
    else
        hipLaunchKernelGGL(ndvm_replay<S>, grid, block, smem, stream, A, d_table, single);
    return hipGetLastError();
}

}  // namespace

// Slot counts the kernel is built for (micro-ops per instruction).
bool slots_supported(uint32_t S) { return S == 1 || S == 2 || S == 4; }

hipError_t launch_replay(const LaunchArgs &A, const ProgStatic *d_table, const ProgStatic &single, uint32_t n_prog,
                         uint32_t r_lds, int variant, uint32_t slots, hipStream_t stream) {
    switch (slots) {
    case 4: return launch_s<4>(A, d_table, single, n_prog, r_lds, variant, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace ndvm
