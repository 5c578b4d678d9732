// Replay kernel: forward replay and reverse sweep of a scheduled tape, one
// lane (parameter vector) per GPU thread (Section 3.5: one structural walk,
// numeric payloads widened over the batch axis).
//
// Every instruction is wave-uniform: the opcode and operand words of the
// device program end up in scalar registers, so all 64 lanes of a wave follow
// the same control and branch only on uniform values; per-lane numeric branches
// were turned into selects by the trace producer.  Lane registers live in LDS
// (register r of thread t at lds[r*64 + t], conflict-free 8-byte accesses)
// and, beyond R_lds, in a lane-contiguous workspace area, so every global
// access of a wave is one coalesced 512-byte row.  Small matrices (up to 4x4)
// are loaded into VGPR arrays by fully unrolled code and multiplied with
// fused multiply-add chains; nothing here is a dense contraction, so no
// matrix cores are used.
//
#include <hip/hip_runtime.h>

#include <mutex>

#include "isa.h"
#include "replay.h"

namespace ndvm {
namespace {

// Lane context on the GPU: register r of thread t at lds[r*64 + t] when
// r < r_lds, else in the workspace spill rows; all addressing lane-contiguous.
// Every pointer carries its address space so that LDS, global and uniform
// (scalar) accesses compile to ds_*, global_* and s_load instructions.
#define AS_LDS __attribute__((address_space(3)))
#define AS_GLOBAL __attribute__((address_space(1)))
#define AS_CONST __attribute__((address_space(4)))

template <bool kSpill>
struct DevCtx {
    AS_LDS double *lds;
    AS_GLOBAL double *spill;
    const AS_CONST double *consts;
    const AS_CONST double *obs;
    const AS_GLOBAL double *params;
    AS_GLOBAL double *loss, *grad, *ckpt;
    int64_t lane, lc, Lpad, ld_p, ld_g;
    uint32_t r_lds;
    uint32_t lane_addr;   // LDS byte address of this thread's register 0
    uint32_t k512;        // 512 (bytes between consecutive registers), kept in a VGPR
    int t;
    bool active;

    __device__ __forceinline__ static uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }
    // every thread of the workgroup (one wave, all threads active) has b
    __device__ __forceinline__ static bool all(bool b) { return __all(b); }
    // Program chunks: thread t loads words 4t..4t+3 of a 32-instruction
    // chunk (one coalesced 1 KiB load per wave), so instruction i lies in
    // threads 2i (words 0-3) and 2i+1 (words 4-7) and v_readlane moves its
    // words into scalar registers.  The chunk in flight sits in registers
    // that nothing reads until the whole current chunk has executed.
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    using Chunk = u32x4;
    __device__ __forceinline__ Chunk load_chunk(const uint32_t *p) const {
        return ((const AS_GLOBAL u32x4 *)(p))[t];
    }
    struct Words {
        Chunk ch;
        int l0;
        __device__ __forceinline__ uint32_t operator[](int k) const {
            const int lane = l0 + (k >> 2);
            switch (k & 3) {
            case 0: return uint32_t(__builtin_amdgcn_readlane(int(ch.x), lane));
            case 1: return uint32_t(__builtin_amdgcn_readlane(int(ch.y), lane));
            case 2: return uint32_t(__builtin_amdgcn_readlane(int(ch.z), lane));
            default: return uint32_t(__builtin_amdgcn_readlane(int(ch.w), lane));
            }
        }
    };
    __device__ __forceinline__ static Words instr(const Chunk &ch, uint32_t i) { return Words{ch, int(2 * i)}; }
    __device__ __forceinline__ static uint32_t aux_word(const uint32_t *aux, uint32_t i) {
        return ((const AS_CONST uint32_t *)(aux))[i];
    }
    __device__ __forceinline__ double ld(uint32_t r) const {
        if (!kSpill || r < r_lds) return lds[r * 64u + t];
        return spill[int64_t(r - r_lds) * Lpad + lane];
    }
    __device__ __forceinline__ double ld_raw(uint32_t r) const { return ld(r); }
    // Register named by the low (hi = 0) or high half of a scalar word.  In
    // LDS its byte address is half * 512 + lane_addr, formed by one
    // v_mad_u32_u16 that reads the half straight from the scalar word.
    __device__ __forceinline__ AS_LDS double *half_ptr(uint32_t word, int hi) const {
        uint32_t addr;
        if (hi)
            asm("v_mad_u32_u16 %0, %1, %2, %3 op_sel:[1,0,0,0]" : "=v"(addr) : "s"(word), "v"(k512), "v"(lane_addr));
        else
            asm("v_mad_u32_u16 %0, %1, %2, %3" : "=v"(addr) : "s"(word), "v"(k512), "v"(lane_addr));
        return (AS_LDS double *)(size_t)addr;
    }
    __device__ __forceinline__ double ldh(uint32_t word, int hi) const {
        if (kSpill) return ld(hi ? word >> 16 : word & 0xFFFFu);
        return *half_ptr(word, hi);
    }
    __device__ __forceinline__ double ldh_raw(uint32_t word, int hi) const { return ldh(word, hi); }
    __device__ __forceinline__ void sth(uint32_t word, int hi, double v) const {
        if (kSpill)
            st(hi ? word >> 16 : word & 0xFFFFu, v);
        else
            *half_ptr(word, hi) = v;
    }
    __device__ __forceinline__ void st(uint32_t r, double v) const {
        if (!kSpill || r < r_lds)
            lds[r * 64u + t] = v;
        else
            spill[int64_t(r - r_lds) * Lpad + lane] = v;
    }
    __device__ __forceinline__ double konst(uint32_t i) const { return consts[i]; }
    __device__ __forceinline__ double obsv(uint32_t i) const { return obs[i]; }
    __device__ __forceinline__ double param(uint32_t p) const { return params[lc * ld_p + p]; }
    __device__ __forceinline__ void store_loss(double v) const {
        if (active) loss[lane] = v;
    }
    __device__ __forceinline__ void store_grad(uint32_t p, double v) const {
        if (active) grad[lane * ld_g + p] = v;
    }
    __device__ __forceinline__ void ckpt_st(uint32_t row, double v) const { ckpt[int64_t(row) * Lpad + lane] = v; }
    __device__ __forceinline__ double ckpt_ld(uint32_t row) const { return ckpt[int64_t(row) * Lpad + lane]; }
};

template <class T>
__device__ __forceinline__ AS_GLOBAL T *gptr(T *p) {
    return (AS_GLOBAL T *)(p);
}
template <class T>
__device__ __forceinline__ const AS_CONST T *cptr(const T *p) {
    return (const AS_CONST T *)(p);
}

}  // namespace

template <bool kSpill>
__device__ __forceinline__ void replay_body(const LaunchArgs &A, const ProgStatic *__restrict__ table,
                                            const ProgStatic &single) {
    extern __shared__ double lds_regs[];
    const uint32_t q = blockIdx.y;
    const ProgStatic D = table ? table[q] : single;
    DevCtx<kSpill> c;
    c.t = threadIdx.x;
    c.lane = int64_t(blockIdx.x) * 64 + c.t;
    c.active = c.lane < A.L;
    c.lc = c.active ? c.lane : A.L - 1;
    c.lds = (AS_LDS double *)lds_regs;
    c.lane_addr = uint32_t(size_t(c.lds + c.t));
    c.k512 = 512u;
    c.spill = gptr(A.ws + int64_t(D.spill_row0) * A.Lpad);
    c.ckpt = gptr(A.ws + int64_t(D.ckpt_row0) * A.Lpad);
    c.consts = cptr(D.consts);
    c.obs = cptr(A.obs);
    c.params = gptr(A.params + int64_t(q) * A.prog_stride_p);
    c.loss = gptr(A.loss + int64_t(q) * A.L);
    c.grad = gptr(A.grad + int64_t(q) * A.prog_stride_g);
    c.Lpad = A.Lpad;
    c.ld_p = A.ld_p;
    c.ld_g = A.ld_g;
    c.r_lds = D.r_lds;
    replay::run(c, D.prog, D.aux);
}

// All lane registers in LDS (the usual case: the scheduler fits the register
// file to the launch's LDS budget).
extern "C" __global__ void __launch_bounds__(64)
ndvm_replay(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    replay_body<false>(A, table, single);
}

// Registers beyond r_lds spill to lane-contiguous workspace rows.
extern "C" __global__ void __launch_bounds__(64)
ndvm_replay_spill(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    replay_body<true>(A, table, single);
}

// Many programs in one launch, only some of which spill: each workgroup takes
// the variant its program needs, so one spilling program does not slow the
// others down.
extern "C" __global__ void __launch_bounds__(64)
ndvm_replay_per_program(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    if (table[blockIdx.y].spills)
        replay_body<true>(A, table, single);
    else
        replay_body<false>(A, table, single);
}

hipError_t launch_replay(const LaunchArgs &A, const ProgStatic *d_table, const ProgStatic &single, uint32_t n_prog,
                         uint32_t r_lds, int variant, hipStream_t stream) {
    static std::once_flag once[64];
    int dev = 0;
    (void)hipGetDevice(&dev);
    std::call_once(once[dev & 63], [dev]() {
        int max_smem = 0;
        (void)hipDeviceGetAttribute(&max_smem, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&ndvm_replay),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&ndvm_replay_spill),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(&ndvm_replay_per_program),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
    });
    dim3 grid(uint32_t(A.Lpad / 64), n_prog), block(64);
    size_t smem = size_t(r_lds) * 64 * sizeof(double);
    if (variant == kPerProgram && d_table)
        hipLaunchKernelGGL(ndvm_replay_per_program, grid, block, smem, stream, A, d_table, single);
    else if (variant == kSpill || variant == kPerProgram)
        hipLaunchKernelGGL(ndvm_replay_spill, grid, block, smem, stream, A, d_table, single);
    else
        hipLaunchKernelGGL(ndvm_replay, grid, block, smem, stream, A, d_table, single);
    return hipGetLastError();
}

}  // namespace ndvm
