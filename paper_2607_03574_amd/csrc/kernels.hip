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

#include "../../include/ndvm.h"
#include "slot.h"
#include "slot_exec.h"

namespace ndvm {
namespace {

#define AS_LDS __attribute__((address_space(3)))
#define AS_GLOBAL __attribute__((address_space(1)))

template <int S, bool kSpill>
struct DevCtx {
    static constexpr int LW = 64 / S;                        // lanes per wave
    static constexpr uint32_t kStride = LW * sizeof(double); // bytes between consecutive registers
    AS_GLOBAL double *spill;
    const AS_GLOBAL double *consts, *obs, *params;
    AS_GLOBAL double *loss, *grad, *ckpt;
    int64_t lane, lc, Lpad, ld_p, ld_g;
    uint32_t r_lds, lane_addr, slot_;
    bool active;

    __device__ __forceinline__ uint32_t slot() const { return slot_; }
    // registers are named by their LDS byte address in this thread's lane
    __device__ __forceinline__ static uint32_t adv(uint32_t h, uint32_t n) { return h + n * kStride; }
    __device__ __forceinline__ double ld(uint32_t h) const {
        if (!kSpill) return *(AS_LDS double *)(size_t)h;
        const uint32_t r = (h - lane_addr) / kStride;
        if (r < r_lds) return *(AS_LDS double *)(size_t)h;
        return spill[int64_t(r - r_lds) * Lpad + lane];
    }
    __device__ __forceinline__ double ld_raw(uint32_t h) const { return ld(h); }
    __device__ __forceinline__ void st(uint32_t h, double v) const {
        if (!kSpill) {
            *(AS_LDS double *)(size_t)h = v;
            return;
        }
        const uint32_t r = (h - lane_addr) / kStride;
        if (r < r_lds)
            *(AS_LDS double *)(size_t)h = v;
        else
            spill[int64_t(r - r_lds) * Lpad + lane] = v;
    }
    __device__ __forceinline__ double obsv(uint32_t i) const { return obs[i]; }
    __device__ __forceinline__ double konst(uint32_t i) const { return consts[i]; }
    __device__ __forceinline__ double param(uint32_t p) const { return params[lc * ld_p + p]; }
    __device__ __forceinline__ static void settle(double v) { asm volatile("" ::"v"(v)); }
    __device__ __forceinline__ static void check_written(uint32_t) {}
    // SKIP: the next n instructions are skipped when every lane of the wave
    // decides the branch the other way (a ballot over the wave's threads; the
    // threads of a lane's slots hold the same predicate)
    mutable uint32_t skip = 0;
    __device__ __forceinline__ void skip_arm(bool then_taken, uint32_t imm) const {
        const uint64_t m = __ballot(then_taken);
        const bool else_arm = (imm >> slot::kSkipSideShift) & 1u;
        if (else_arm ? m == ~uint64_t(0) : m == 0) skip = imm & slot::kSkipCountMask;
    }
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
__device__ __forceinline__ uint32_t lane_word(uint32_t v, uint32_t lane) {
    return uint32_t(__builtin_amdgcn_readlane(int(v), int(lane)));
}

// A copy of a wave-uniform value that the compiler cannot see through.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
    asm("" : "+s"(v));
    return v;
}

// LDS addresses of the four register fields of instruction P of the chunk
// word `ch`: each is the broadcast byte offset plus this thread's lane
// address, one DPP-sourced add per field.  A DPP read of a VGPR that a VALU
// op wrote needs two wait states between them (the s_nop, kept where the
// chunk word may just have been copied into place); no VALU op of this
// kernel writes EXEC.  Volatile: the decode of the next instruction stays
// where it is placed, in the shadow of the current instruction's loads.
struct Fields {
    uint32_t a, x, y, z;
};
template <int P, bool kNop>
__device__ __forceinline__ void decode(uint32_t ch, uint32_t la, Fields &f) {
    if constexpr (kNop) {
        asm volatile(
            "s_nop 1\n\t"
            "v_add_u32_dpp %0, %4, %5 row_newbcast:%6 row_mask:0xf bank_mask:0xf\n\t"
            "v_add_u32_dpp %1, %4, %5 row_newbcast:%7 row_mask:0xf bank_mask:0xf\n\t"
            "v_add_u32_dpp %2, %4, %5 row_newbcast:%8 row_mask:0xf bank_mask:0xf\n\t"
            "v_add_u32_dpp %3, %4, %5 row_newbcast:%9 row_mask:0xf bank_mask:0xf"
            : "=&v"(f.a), "=&v"(f.x), "=&v"(f.y), "=&v"(f.z)
            : "v"(ch), "v"(la), "i"(4 * P), "i"(4 * P + 1), "i"(4 * P + 2), "i"(4 * P + 3));
    } else {
        asm volatile(
            "v_add_u32_dpp %0, %4, %5 row_newbcast:%6 row_mask:0xf bank_mask:0xf\n\t"
            "v_add_u32_dpp %1, %4, %5 row_newbcast:%7 row_mask:0xf bank_mask:0xf\n\t"
            "v_add_u32_dpp %2, %4, %5 row_newbcast:%8 row_mask:0xf bank_mask:0xf\n\t"
            "v_add_u32_dpp %3, %4, %5 row_newbcast:%9 row_mask:0xf bank_mask:0xf"
            : "=&v"(f.a), "=&v"(f.x), "=&v"(f.y), "=&v"(f.z)
            : "v"(ch), "v"(la), "i"(4 * P), "i"(4 * P + 1), "i"(4 * P + 2), "i"(4 * P + 3));
    }
}

// Payload of instruction P of a chunk: register fields as LDS addresses,
// the header supplies the immediate and this slot's flags; loaded() runs
// the decode of the next instruction (the handlers call it once, between
// their reads and their arithmetic).
template <int P, class N>
struct ChunkPayload {
    uint32_t ha, hx, hy, hz, ch, hdr, slot;
    N *nx;
    __device__ __forceinline__ uint32_t a() const { return ha; }
    __device__ __forceinline__ uint32_t x() const { return hx; }
    __device__ __forceinline__ uint32_t y() const { return hy; }
    __device__ __forceinline__ uint32_t z() const { return hz; }
    __device__ __forceinline__ uint32_t ix() const { return row_word<4 * P + 1>(ch); }
    __device__ __forceinline__ uint32_t imm() const { return hdr >> slot::kImmShift; }
    __device__ __forceinline__ bool first() const { return (hdr >> (slot::kFirstShift + slot)) & 1u; }
    __device__ __forceinline__ void loaded() const { (*nx)(); }
};
// Payload of a cold instruction, words read out
struct Payload {
    uint32_t w[4], hdr, slot, lane_addr;
    __device__ __forceinline__ uint32_t a() const { return w[0] + lane_addr; }
    __device__ __forceinline__ uint32_t x() const { return w[1] + lane_addr; }
    __device__ __forceinline__ uint32_t y() const { return w[2] + lane_addr; }
    __device__ __forceinline__ uint32_t z() const { return w[3] + lane_addr; }
    __device__ __forceinline__ uint32_t ix() const { return w[1]; }
    __device__ __forceinline__ uint32_t imm() const { return hdr >> slot::kImmShift; }
    __device__ __forceinline__ bool first() const { return (hdr >> (slot::kFirstShift + slot)) & 1u; }
};

// Cold micro-ops run out of line: their library code branches per lane, and
// keeping those branches out of the replay loop leaves its hot part free of
// divergent control flow.
template <class C>
__device__ __attribute__((noinline)) void cold_call(const C &c, uint32_t form, Payload p) {
    slotx::exec_cold(c, form, p);
}

// Instruction P of the chunk held in `ch` (one dword per thread), header
// lane hb of `hv`, register fields `f` (decoded by the previous
// instruction); `next` decodes the following instruction.  END and the
// padding after it do nothing: the loop below runs the chunks up to the one
// holding END and stops.
template <int P, bool kSkip, int kOrder, class C, class N>
__device__ __forceinline__ void step(const C &c, uint32_t ch, uint32_t hv, uint32_t hb, const Fields &f, N &next) {
    if (kSkip && c.skip) {   // inside a skipped arm (never holds END)
        --c.skip;
        next();
        return;
    }
    const uint32_t hdr = lane_word(hv, hb);
    const uint32_t form = hdr & slot::kFormMask;
    const ChunkPayload<P, N> p{f.a, f.x, f.y, f.z, ch, hdr, c.slot_, &next};
    // the most frequent forms are tested one by one, each by its own header
    // bit, ahead of the dispatch tree, in the launch's order (DispatchOrder);
    // the first runs straight into the next instruction.  The empty asm
    // hides that the tree's tests are on the same value as the form, so the
    // compiler cannot fold the tests into one balanced tree (which would put
    // every form several compares deep).
    if constexpr (kOrder == slot::kOrderAccMacMsub) {
        if (__builtin_expect((hdr & slot::kAccBit) != 0, 1)) {
            slotx::exec_acc(c, p);
            return;
        }
        if (__builtin_expect((hdr & slot::kMacBit) != 0, 1)) {
            slotx::exec_mac(c, p);
            return;
        }
        if (__builtin_expect((hdr & slot::kMsubBit) != 0, 1)) {
            slotx::exec_msub(c, p);
            return;
        }
    } else if constexpr (kOrder == slot::kOrderMacBlock) {
        if (__builtin_expect((hdr & slot::kMacBit) != 0, 1)) {
            slotx::exec_mac(c, p);
            return;
        }
        if (__builtin_expect((hdr & slot::kBlockBit) != 0, 1)) {
            if (form == slot::DOTB)
                slotx::dot_block<false>(c, p);
            else
                slotx::dot_block<true>(c, p);
            return;
        }
    } else {
        if (__builtin_expect((hdr & slot::kMacBit) != 0, 1)) {
            slotx::exec_mac(c, p);
            return;
        }
        if (__builtin_expect((hdr & slot::kAccBit) != 0, 1)) {
            slotx::exec_acc(c, p);
            return;
        }
    }
    const uint32_t f2 = opaque(form);
    if (f2 < slot::HOT_END) {
        slotx::exec_hot(c, f2, p);
        return;
    }
    next();
    if (f2 == slot::END) return;
    cold_call(c, f2,
              Payload{{row_word<4 * P>(ch), row_word<4 * P + 1>(ch), row_word<4 * P + 2>(ch), row_word<4 * P + 3>(ch)},
                      hdr, c.slot_, c.lane_addr});
}

// Execute a slot program through the chunk holding END: the four
// instructions of each chunk in straight-line code, chunk c + 2 requested
// when chunk c starts, the headers of 64 chunks at a time (four per thread)
// with the next group in flight (the program is padded for these
// read-aheads: the chunk holding END is followed by kFetchAhead chunks,
// which is how the chunk count is known, and instructions after END are END
// too).
template <bool kSkip, int kOrder, int S, bool kSpill>
__device__ __forceinline__ void run(const DevCtx<S, kSpill> &c, const uint32_t *prog, uint32_t hdr_off) {
    static_assert(slot::kChunk == 4 && slot::kFetchAhead == 2 && slot::kHeaderGroup == 256,
                  "the fetch below reads four-instruction chunks two ahead and the headers of 64 chunks a group");
    using Hdr4 = uint32_t __attribute__((ext_vector_type(4)));
    const AS_GLOBAL uint32_t *pc = (const AS_GLOBAL uint32_t *)prog + threadIdx.x;
    const AS_GLOBAL Hdr4 *ph = (const AS_GLOBAL Hdr4 *)((const AS_GLOBAL uint32_t *)prog + hdr_off) + threadIdx.x;
    constexpr uint32_t W = slot::kChunkWords;
    uint32_t cur = pc[0], n1 = pc[W];
    Hdr4 hv = ph[0], hn = ph[64];
    const uint32_t n_chunks = hdr_off / W - slot::kFetchAhead;
    const uint32_t la = c.lane_addr;
    Fields f0, f1, f2, f3;
    decode<0, true>(cur, la, f0);
    for (uint32_t chunk = 0; chunk < n_chunks; ++chunk) {
        pc += W;
        const uint32_t n2 = pc[W];
        const uint32_t hb = chunk & 63u;
        auto d1 = [&] { decode<1, true>(cur, la, f1); };
        auto d2 = [&] { decode<2, false>(cur, la, f2); };
        auto d3 = [&] { decode<3, false>(cur, la, f3); };
        auto d0 = [&] { decode<0, true>(n1, la, f0); };   // instruction 0 of the next chunk
        step<0, kSkip, kOrder>(c, cur, hv.x, hb, f0, d1);
        step<1, kSkip, kOrder>(c, cur, hv.y, hb, f1, d2);
        step<2, kSkip, kOrder>(c, cur, hv.z, hb, f2, d3);
        step<3, kSkip, kOrder>(c, cur, hv.w, hb, f3, d0);
        cur = n1;
        n1 = n2;
        if (hb == 63u) {
            ph += 64;
            hv = hn;
            hn = ph[64];
        }
    }
}

}  // namespace

// Program and lane block of this workgroup: the grid's (y, x), or the work
// item the launch's table gives it (false: none).
__device__ __forceinline__ bool work_item(const LaunchArgs &A, uint32_t &q, uint32_t &bx) {
    if (!A.wg_items) {
        q = blockIdx.y;
        bx = blockIdx.x;
        return true;
    }
    const uint64_t it = A.wg_items[blockIdx.x];
    q = uint32_t(it >> 32);
    bx = uint32_t(it);
    return it != ~uint64_t(0);
}

template <int S, bool kSpill, bool kSkip, int kOrder>
__device__ __forceinline__ void replay_body(const LaunchArgs &A, const ProgStatic *__restrict__ table,
                                            const ProgStatic &single, uint32_t q, uint32_t bx) {
    extern __shared__ double lds_regs[];
    constexpr int LW = 64 / S;
    const ProgStatic D = table ? table[q] : single;
    DevCtx<S, kSpill> c;
    const int t = threadIdx.x, l = t % LW;
    c.slot_ = uint32_t(t / LW);
    c.lane = int64_t(bx) * LW + l;
    c.active = c.lane < A.L;
    c.lc = c.active ? c.lane : A.L - 1;
    const AS_GLOBAL double *obs_row = (const AS_GLOBAL double *)A.obs;
    if (A.n_points > 0) {   // flattened data axis: parameter row and data point of the lane
        obs_row += (c.lc % A.n_points) * A.obs_stride;
        c.lc = c.lc / A.n_points;
    }
    c.lane_addr = uint32_t(size_t((AS_LDS double *)lds_regs + l));
    c.spill = (AS_GLOBAL double *)(A.ws + int64_t(D.spill_row0) * A.Lpad);
    c.ckpt = (AS_GLOBAL double *)(A.ws + int64_t(D.ckpt_row0) * A.Lpad);
    c.consts = (const AS_GLOBAL double *)D.consts;
    c.obs = obs_row;
    c.params = (const AS_GLOBAL double *)(A.params + int64_t(q) * A.prog_stride_p);
    c.loss = (AS_GLOBAL double *)(A.loss + int64_t(q) * A.L);
    c.grad = (AS_GLOBAL double *)(A.grad + int64_t(q) * A.prog_stride_g);
    c.Lpad = A.Lpad;
    c.ld_p = A.ld_p;
    c.ld_g = A.ld_g;
    c.r_lds = D.r_lds;
    run<kSkip, kOrder>(c, D.prog, D.hdr_off);
}

// All lane registers in LDS (the usual case: the scheduler fits the register
// file to the launch's LDS budget).  kSkip: the program has skippable branch
// arms (every instruction then tests the skip counter first).  kOrder: the
// order of the form tests (DispatchOrder).
template <int S, bool kSkip, int kOrder>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4)))
ndvm_replay(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    uint32_t q, bx;
    if (work_item(A, q, bx)) replay_body<S, false, kSkip, kOrder>(A, table, single, q, bx);
}

// Registers beyond r_lds spill to lane-contiguous workspace rows.
template <int S>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4)))
ndvm_replay_spill(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    uint32_t q, bx;
    if (work_item(A, q, bx)) replay_body<S, true, true, slot::kOrderMacAcc>(A, table, single, q, bx);
}

// Many programs in one launch, only some of which spill: each workgroup takes
// the variant its program needs, so one spilling program does not slow the
// others down.
template <int S, bool kSkip>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4)))
ndvm_replay_per_program(LaunchArgs A, const ProgStatic *__restrict__ table, ProgStatic single) {
    uint32_t q, bx;
    if (!work_item(A, q, bx)) return;
    if (table[q].spills)
        replay_body<S, true, true, slot::kOrderMacAcc>(A, table, single, q, bx);
    else
        replay_body<S, false, kSkip, slot::kOrderMacAcc>(A, table, single, q, bx);
}

namespace {

template <int S, bool kSkip>
void launch_ordered(dim3 grid, dim3 block, size_t smem, hipStream_t stream, const LaunchArgs &A,
                    const ProgStatic *d_table, const ProgStatic &single, int order) {
    if (order == slot::kOrderAccMacMsub)
        hipLaunchKernelGGL((ndvm_replay<S, kSkip, slot::kOrderAccMacMsub>), grid, block, smem, stream, A, d_table,
                           single);
    else if (order == slot::kOrderMacBlock)
        hipLaunchKernelGGL((ndvm_replay<S, kSkip, slot::kOrderMacBlock>), grid, block, smem, stream, A, d_table,
                           single);
    else
        hipLaunchKernelGGL((ndvm_replay<S, kSkip, slot::kOrderMacAcc>), grid, block, smem, stream, A, d_table,
                           single);
}

template <int S>
hipError_t launch_s(const LaunchArgs &A, const ProgStatic *d_table, const ProgStatic &single, uint32_t n_prog,
                    uint32_t r_lds, int variant, bool skips, int order, hipStream_t stream) {
    static std::once_flag once[64];
    int dev = 0;
    (void)hipGetDevice(&dev);
    std::call_once(once[dev & 63], [dev]() {
        int max_smem = 0;
        (void)hipDeviceGetAttribute(&max_smem, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
        for (const void *f : {reinterpret_cast<const void *>(&ndvm_replay<S, false, slot::kOrderMacAcc>),
                              reinterpret_cast<const void *>(&ndvm_replay<S, true, slot::kOrderMacAcc>),
                              reinterpret_cast<const void *>(&ndvm_replay<S, false, slot::kOrderAccMacMsub>),
                              reinterpret_cast<const void *>(&ndvm_replay<S, true, slot::kOrderAccMacMsub>),
                              reinterpret_cast<const void *>(&ndvm_replay<S, false, slot::kOrderMacBlock>),
                              reinterpret_cast<const void *>(&ndvm_replay<S, true, slot::kOrderMacBlock>),
                              reinterpret_cast<const void *>(&ndvm_replay_spill<S>),
                              reinterpret_cast<const void *>(&ndvm_replay_per_program<S, false>),
                              reinterpret_cast<const void *>(&ndvm_replay_per_program<S, true>)})
            (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, max_smem);
    });
    constexpr int LW = 64 / S;
    dim3 grid = A.wg_items ? dim3(A.n_wg) : dim3(uint32_t((A.L + LW - 1) / LW), n_prog), block(64);
    size_t smem = size_t(r_lds) * LW * sizeof(double);
    if (variant == kPerProgram && d_table) {
        if (skips)
            hipLaunchKernelGGL((ndvm_replay_per_program<S, true>), grid, block, smem, stream, A, d_table, single);
        else
            hipLaunchKernelGGL((ndvm_replay_per_program<S, false>), grid, block, smem, stream, A, d_table, single);
    } else if (variant == kSpill || variant == kPerProgram) {
        hipLaunchKernelGGL(ndvm_replay_spill<S>, grid, block, smem, stream, A, d_table, single);
    } else if (skips) {
        launch_ordered<S, true>(grid, block, smem, stream, A, d_table, single, order);
    } else {
        launch_ordered<S, false>(grid, block, smem, stream, A, d_table, single, order);
    }
    return hipGetLastError();
}

}  // namespace

// Reduction of the flattened data axis: loss[l] = scale * left fold over the
// points in ascending order of term[l*N + i], and likewise every gradient
// entry; one thread per (parameter row, output), consecutive threads on the
// outputs of one row.  Each thread reads its own N terms in order (the fold
// order is part of the result's definition).
__global__ void __launch_bounds__(256) ndvm_fold_points(const double *__restrict__ term,
                                                        const double *__restrict__ tgrad, int64_t L, int64_t N,
                                                        int64_t P, double scale, double *__restrict__ loss,
                                                        double *__restrict__ grad, int64_t ld_g) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= L * (P + 1)) return;
    const int64_t l = i / (P + 1), k = i % (P + 1);
    double acc = 0.0;
    if (k == P) {
        const double *t = term + l * N;
        for (int64_t j = 0; j < N; ++j) acc = acc + t[j];
        loss[l] = acc * scale;
    } else {
        const double *g = tgrad + l * N * P + k;
        for (int64_t j = 0; j < N; ++j) acc = acc + g[j * P];
        grad[l * ld_g + k] = acc * scale;
    }
}

hipError_t launch_fold_points(const double *term, const double *tgrad, int64_t L, int64_t N, int64_t P,
                              double scale, double *loss, double *grad, int64_t ld_g, hipStream_t stream) {
    const int64_t n = L * (P + 1);
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(ndvm_fold_points, dim3(uint32_t((n + 255) / 256)), dim3(256), 0, stream, term, tgrad, L, N,
                       P, scale, loss, grad, ld_g);
    return hipGetLastError();
}

// Slot counts the kernel is built for (micro-ops per instruction).
bool slots_supported(uint32_t S) { return S == 4; }

// Static workspace of the allocation-free gradient entry point: checkpoint,
// trash and spill rows of one launch live here instead of in a caller
// workspace.  Each GPU the library runs on holds its own copy from module load
// until the process ends.  Host code never passes `scratch` itself to a
// kernel: in host code the name is a host-side stand-in, not a device
// address; the device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = NDVM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) double scratch[kScratchBytes / sizeof(double)];

size_t scratch_bytes() { return kScratchBytes; }

// Device address of `scratch` on the current device, looked up on the first
// call per device (with that device current) and cached.
hipError_t scratch_address(void **out) {
    static std::mutex mu;
    static void *addr[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (!addr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!ptr) return hipErrorInvalidSymbol;
        addr[dev] = ptr;
    }
    *out = addr[dev];
    return hipSuccess;
}

hipError_t launch_replay(const LaunchArgs &A, const ProgStatic *d_table, const ProgStatic &single, uint32_t n_prog,
                         uint32_t r_lds, int variant, bool skips, int order, uint32_t slots,
                         hipStream_t stream) {
    switch (slots) {
    case 4: return launch_s<4>(A, d_table, single, n_prog, r_lds, variant, skips, order, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace ndvm
