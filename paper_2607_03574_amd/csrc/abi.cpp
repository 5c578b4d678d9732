// C ABI of libndvm: tape handles, device programs, workspace sizing and the
// launch of the replay kernel.  Every entry point validates its arguments
// before enqueuing anything and converts exceptions into status codes.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <memory>
#include <mutex>
#include <thread>
#include <new>

#include "common.h"
#include "slot.h"
#include "sched.h"

namespace ndvm {
hipError_t launch_replay(const LaunchArgs &A, const ProgStatic *d_table, const ProgStatic &single, uint32_t n_prog,
                         uint32_t r_lds, int variant, bool skips, int order, uint32_t slots,
                         hipStream_t stream);
bool slots_supported(uint32_t S);
size_t scratch_bytes();
hipError_t launch_fold_points(const double *term, const double *tgrad, int64_t L, int64_t N, int64_t P,
                              double scale, double *loss, double *grad, int64_t ld_g, hipStream_t stream);
hipError_t scratch_address(void **out);
struct AdamArgs {
    double *p;
    const double *g;
    double *m, *v;
    int64_t L, P, ld_p, ld_g;
    double lr, b1, b2, eps, c1, c2;
};
hipError_t launch_adam(const AdamArgs &a, hipStream_t stream);
}

using namespace ndvm;

namespace {

struct DeviceProps {
    int cus = 256;
    size_t lds_per_cu = 160 * 1024;
    size_t lds_per_block = 64 * 1024;
};

std::mutex g_props_mu;
std::map<int, DeviceProps> g_props;

ndvm_status device_props(DeviceProps *out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        set_error("hipGetDevice failed");
        return NDVM_E_DEVICE;
    }
    std::lock_guard<std::mutex> lk(g_props_mu);
    auto it = g_props.find(dev);
    if (it == g_props.end()) {
        DeviceProps p;
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) p.cus = v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && v > 0)
            p.lds_per_block = size_t(v);
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) == hipSuccess && v > 0)
            p.lds_per_cu = size_t(v);
        it = g_props.emplace(dev, p).first;
    }
    *out = it->second;
    return NDVM_OK;
}

constexpr uint32_t kMaxWavesPerCuTarget = 16;
// programs per many-program launch (the grid's y extent)
constexpr int kMaxProgPerLaunch = 65535;

// Micro-ops per instruction (threads per lane) of a launch: 4 slots (16
// lanes per wave).  Fewer slots would leave fewer unused slots per
// instruction, but give each lane a quarter or half the LDS registers at the
// same wave count (measured: the program population at 1 slot spills and
// runs 3x slower), so the format keeps 4.
uint32_t choose_slots(const DeviceProps &p, int64_t L, int64_t n_prog) {
    (void)p;
    (void)L;
    (void)n_prog;
    return slot::kMaxSlots;
}
// bytes of one register of one wave (64/S lanes)
size_t reg_bytes(uint32_t S) { return size_t(64 / S) * sizeof(double); }
int64_t waves_of(int64_t L, int64_t n_prog, uint32_t S) { return (L + 64 / S - 1) / (64 / S) * n_prog; }

// Registers per lane that may live in LDS for a launch of `waves` waves:
// enough waves resident per CU to cover the launch (at most 16), LDS split
// evenly between them.
uint32_t reg_budget(const DeviceProps &p, int64_t waves, uint32_t S) {
    int64_t per_cu = (waves + p.cus - 1) / p.cus;
    per_cu = std::max<int64_t>(1, std::min<int64_t>(per_cu, kMaxWavesPerCuTarget));
    size_t bytes = std::min(p.lds_per_cu / size_t(per_cu), p.lds_per_block);
    return uint32_t(bytes / reg_bytes(S));
}

struct DevProg {
    Schedule meta;          // host copy of counts (code vector released)
    void *buf = nullptr;    // device: code | consts
    const uint32_t *code = nullptr;
    const double *consts = nullptr;
    ~DevProg() {
        if (buf) (void)hipFree(buf);
    }
};

std::atomic<uint64_t> g_next_id{1};

}  // namespace

struct ndvm_tape {
    uint64_t id = 0;
    Tape tape;
    uint64_t tape_bytes = 0;
    uint32_t n_selects = 0;
    int policy = NDVM_POLICY_RECOMPUTE;
    bool arms = false;   // NDVM_BRANCH_SKIP: branch arms behind wave skip tests
    std::mutex mu;
    std::map<uint32_t, std::unique_ptr<DevProg>> fwd;    // keyed by slot count
    std::map<uint64_t, std::unique_ptr<DevProg>> grad;   // keyed by (slot count, register budget)
};

namespace {

ndvm_status upload_program(Schedule &&S, const Tape &t, hipStream_t stream, std::unique_ptr<DevProg> *out) {
    // the kernel fetches whole chunks and reads two chunks past the one that
    // holds END
    const uint64_t end_at = uint64_t(S.n_instr) - 1;   // index of the END instruction
    if (S.hdr_off != uint64_t(S.n_chunks) * slot::kChunkWords || S.n_instr == 0 ||
        end_at / slot::kChunk + 1 + slot::kFetchAhead > S.n_chunks ||
        S.hdr_off + (end_at / slot::kHeaderGroup + 1 + slot::kFetchAhead) * slot::kHeaderGroup > S.code.size() ||
        (S.code[S.hdr_off + end_at] & slot::kFormMask) != slot::END) {
        set_error("internal: device program is not padded to the fetch chunks");
        return NDVM_E_TAPE;
    }
    auto dp = std::make_unique<DevProg>();
    size_t code_b = S.code.size() * 4, con_b = S.consts.size() * 8;
    size_t con_off = (code_b + 255) / 256 * 256;
    size_t total = con_off + std::max<size_t>(con_b, 8);
    if (hipMalloc(&dp->buf, total) != hipSuccess) {
        (void)hipGetLastError();
        dp->buf = nullptr;
        set_error("hipMalloc of the device program failed");
        return NDVM_E_NOMEM;
    }
    std::vector<uint8_t> host(total, 0);
    std::memcpy(host.data(), S.code.data(), code_b);
    if (con_b) std::memcpy(host.data() + con_off, S.consts.data(), con_b);
    if (hipMemcpyAsync(dp->buf, host.data(), total, hipMemcpyHostToDevice, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess) {
        set_error("copy of the device program failed");
        return NDVM_E_DEVICE;
    }
    dp->code = reinterpret_cast<const uint32_t *>(dp->buf);
    dp->consts = reinterpret_cast<const double *>(static_cast<uint8_t *>(dp->buf) + con_off);
    S.code.clear();
    S.code.shrink_to_fit();
    dp->meta = std::move(S);
    *out = std::move(dp);
    (void)t;
    return NDVM_OK;
}

// Schedule a program, turning scheduler limits into a status.
template <class F>
ndvm_status scheduled(F f, Schedule *out) {
    try {
        *out = f();
    } catch (const std::length_error &e) {
        set_error(std::string("program too large for the device format: ") + e.what());
        return NDVM_E_UNSUPPORTED;
    }
    return NDVM_OK;
}

// Device program of `tape` for gradient launches with S slots and register
// budget b.  Scheduling and the program's upload happen only in the sizing
// calls (build = true); a compute call finds the program or fails, so it
// never schedules on the host or waits for a copy.
Schedule schedule_grad_of(const ndvm_tape *tape, uint32_t S, uint32_t b) {
    return schedule_grad(tape->tape, b, S, tape->policy == NDVM_POLICY_SAVE, tape->arms ? kArmMinElems : 0);
}

// `pre`: the schedule, when the caller made it already (many-program sizing
// schedules its programs in parallel).
ndvm_status grad_program(ndvm_tape *tape, uint32_t S, uint32_t b, bool build, DevProg **out,
                         Schedule *pre = nullptr) {
    std::lock_guard<std::mutex> lk(tape->mu);
    const uint64_t key = (uint64_t(S) << 32) | b;
    auto it = tape->grad.find(key);
    if (it == tape->grad.end() && !build) {
        set_error("the tape has no device program for this lane count: size the workspace with "
                  "ndvm_workspace_bytes (ndvm_workspace_bytes_many) for the same lane count first");
        return NDVM_E_ARG;
    }
    if (it == tape->grad.end()) {
        const hipStream_t stream = nullptr;
        Schedule sch;
        if (pre) {
            sch = std::move(*pre);
        } else {
            ndvm_status st = scheduled([&] { return schedule_grad_of(tape, S, b); }, &sch);
            if (st != NDVM_OK) return st;
        }
        ndvm_status st;
        std::unique_ptr<DevProg> dp;
        st = upload_program(std::move(sch), tape->tape, stream, &dp);
        if (st != NDVM_OK) return st;
        it = tape->grad.emplace(key, std::move(dp)).first;
    }
    *out = it->second.get();
    return NDVM_OK;
}

// Schedules of the programs among `tapes` that have no device program for
// (S, b) yet, made on all host threads (each program's schedule is
// independent of the others); the uploads stay with the caller.  On a
// failure the first failing program's status and message are returned.
ndvm_status schedule_many(const ndvm_tape *const *tapes, int n_prog, uint32_t S, uint32_t b,
                          std::map<const ndvm_tape *, Schedule> *out) {
    const uint64_t key = (uint64_t(S) << 32) | b;
    std::vector<const ndvm_tape *> todo;
    for (int q = 0; q < n_prog; ++q) {
        ndvm_tape *t = const_cast<ndvm_tape *>(tapes[q]);
        std::lock_guard<std::mutex> lk(t->mu);
        if (!t->grad.count(key) && !out->count(t)) {
            out->emplace(t, Schedule{});
            todo.push_back(t);
        }
    }
    if (todo.empty()) return NDVM_OK;
    std::vector<Schedule> res(todo.size());
    std::vector<ndvm_status> code(todo.size(), NDVM_OK);
    std::vector<std::string> msg(todo.size());
    std::atomic<size_t> next{0};
    auto work = [&]() {
        for (size_t i; (i = next.fetch_add(1)) < todo.size();) {
            try {
                res[i] = schedule_grad_of(todo[i], S, b);
            } catch (const std::length_error &e) {
                code[i] = NDVM_E_UNSUPPORTED;
                msg[i] = std::string("program too large for the device format: ") + e.what();
            } catch (const std::bad_alloc &) {
                code[i] = NDVM_E_NOMEM;
                msg[i] = "out of host memory";
            } catch (const std::exception &e) {
                code[i] = NDVM_E_INTERNAL;
                msg[i] = std::string("internal error: ") + e.what();
            }
        }
    };
    const size_t n_threads = std::min<size_t>(todo.size(), std::max(1u, std::thread::hardware_concurrency()));
    std::vector<std::thread> pool;
    for (size_t k = 1; k < n_threads; ++k) pool.emplace_back(work);
    work();
    for (auto &th : pool) th.join();
    for (size_t i = 0; i < todo.size(); ++i) {
        if (code[i] != NDVM_OK) {
            set_error(msg[i]);
            return code[i];
        }
        (*out)[todo[i]] = std::move(res[i]);
    }
    return NDVM_OK;
}

// Register budget and device program of a single-program gradient launch.
// The budget first sizes LDS so that every wave of the launch is resident
// (at most 16 per CU).  A program whose register file does not fit that
// budget would keep its excess registers in HBM rows; it is scheduled again
// for the budget of as many resident waves per CU as its register file
// leaves room for, and the launch runs in several rounds of waves instead
// (Kalman at 32,768 lanes needs 314 registers against a budget of 160).
// Deterministic in (tape, L), so sizing and compute calls agree.
ndvm_status single_grad_program(ndvm_tape *tape, const DeviceProps &p, int64_t L, uint32_t S, bool build,
                                DevProg **dp, uint32_t *b) {
    *b = reg_budget(p, waves_of(L, 1, S), S);
    ndvm_status st = grad_program(tape, S, *b, build, dp);
    if (st != NDVM_OK || (*dp)->meta.n_regs <= *b) return st;
    const size_t need = size_t((*dp)->meta.n_regs) * reg_bytes(S);
    const size_t per_cu = std::max<size_t>(1, p.lds_per_cu / need);
    const uint32_t b2 = uint32_t(std::min(p.lds_per_cu / per_cu, p.lds_per_block) / reg_bytes(S));
    if (b2 <= *b) return NDVM_OK;
    DevProg *dp2 = nullptr;
    if ((st = grad_program(tape, S, b2, build, &dp2)) != NDVM_OK) return st;
    *dp = dp2;
    *b = b2;
    return NDVM_OK;
}

// Registers of a forward-only program: whatever one workgroup may hold.
uint32_t fwd_budget(uint32_t S) {
    DeviceProps p;
    if (device_props(&p) != NDVM_OK) p = DeviceProps{};
    return uint32_t(p.lds_per_block / reg_bytes(S));
}

// Forward-only device program of `tape` with S slots.
Schedule schedule_forward_of(const ndvm_tape *tape, uint32_t S, uint32_t budget) {
    return schedule_forward(tape->tape, S, budget, tape->arms ? kArmMinElems : 0);
}

// `pre`: the schedule, when the caller made it already.
ndvm_status fwd_program(ndvm_tape *tape, uint32_t S, hipStream_t stream, DevProg **out, Schedule *pre = nullptr) {
    std::lock_guard<std::mutex> lk(tape->mu);
    auto it = tape->fwd.find(S);
    if (it == tape->fwd.end()) {
        Schedule sch;
        ndvm_status st = NDVM_OK;
        if (pre)
            sch = std::move(*pre);
        else
            st = scheduled([&] { return schedule_forward_of(tape, S, fwd_budget(S)); }, &sch);
        if (st != NDVM_OK) return st;
        std::unique_ptr<DevProg> dp;
        st = upload_program(std::move(sch), tape->tape, stream, &dp);
        if (st != NDVM_OK) return st;
        it = tape->fwd.emplace(S, std::move(dp)).first;
    }
    *out = it->second.get();
    return NDVM_OK;
}

int64_t lpad_of(int64_t L) { return (L + 63) / 64 * 64; }

// Workspace rows (fp64 per lane) of one program launched with LDS budget b:
// checkpoint rows, the trash rows that unused slots store to, spill rows.
uint64_t ws_rows(const DevProg &dp, uint32_t b) {
    uint32_t r_lds = std::min(dp.meta.n_regs, b);
    return uint64_t(dp.meta.n_ckpt_rows) + slot::kMaxBlock + (dp.meta.n_regs - r_lds);
}

// Order of the kernel's form tests (slot::DispatchOrder) for a launch whose
// programs hold these instruction counts: the linear adjoint rule first
// (then multiply-add and multiply-subtract) when it outnumbers multiply-add
// and multiply-subtracts are frequent, as in a reverse sweep over ODE steps;
// multiply-add then the block dots when those are a quarter of the
// instructions (small-matrix programs such as a Kalman filter); multiply-add
// then the adjoint rule otherwise.  The first form tested runs without a
// taken branch, every further test costs the forms behind it.
int dispatch_order(uint64_t n_mac, uint64_t n_acc, uint64_t n_msub, uint64_t n_block, uint64_t n_instr) {
    if (n_acc > n_mac && n_msub * 16 >= n_instr) return slot::kOrderAccMacMsub;
    if (n_block * 4 >= n_instr && n_mac >= n_acc) return slot::kOrderMacBlock;
    return slot::kOrderMacAcc;
}
int dispatch_order(const Schedule &m) { return dispatch_order(m.n_mac, m.n_acc, m.n_msub, m.n_block, m.n_instr); }

ndvm_status check_stream_and_launch(const LaunchArgs &A, const ProgStatic *table, const ProgStatic &single,
                                    uint32_t n_prog, uint32_t r_lds, int variant, bool skips, int order,
                                    uint32_t slots, hipStream_t stream) {
    hipError_t e = launch_replay(A, table, single, n_prog, r_lds, variant, skips, order, slots, stream);
    if (e != hipSuccess) {
        set_error(std::string("kernel launch failed: ") + hipGetErrorString(e));
        return NDVM_E_DEVICE;
    }
    return NDVM_OK;
}

// Device tables of ProgStatic for ndvm_grad_many, cached per program set, and
// of per-XCD work items, cached per program set and lane blocks.
std::mutex g_table_mu;
std::map<std::vector<uint64_t>, void *> g_tables;
struct ItemTable {
    void *d = nullptr;   // null: the plain grid
    uint32_t n_wg = 0;
};
std::map<std::vector<uint64_t>, ItemTable> g_items;

// A many-program launch: per-program device programs for the launch's
// register budget, their table of ProgStatic on the device (cached per
// program set) and workspace rows.  With build = false (compute calls)
// nothing is scheduled, allocated or copied: everything must have been
// prepared by ndvm_workspace_bytes_many for the same lane count.
struct ManyLaunch {
    uint32_t S = 0, r_launch = 0;
    int variant = kLdsOnly;
    bool skips = false;     // some program has skippable branch arms
    int order = 0;          // order of the kernel's form tests (dispatch_order over all programs)
    uint64_t rows = 0;
    void *d_table = nullptr;
    const uint64_t *d_items = nullptr;   // work item per workgroup (xcd_items), or null
    uint32_t n_wg = 0;
};

// Work items of a many-program launch laid out per XCD.  Each of MI355X's
// eight XCDs has its own L2, and workgroups are dispatched to them in turn
// (workgroup w to XCD w mod 8), so a program whose waves run on every XCD is
// fetched into every L2.  Whole programs are assigned to XCDs instead,
// longest first to the XCD with the least work so far (the lanes of every
// program are alike, so its instruction count measures its work), and
// workgroup k + 8 i takes the i-th work item (program, lane block) of XCD k:
// an XCD runs the lane blocks of one program one after another.  Used when
// every XCD gets several programs and the largest XCD load is within 5% of
// the mean; otherwise the launch keeps the plain grid.
constexpr uint32_t kXcds = 8;
bool xcd_items(const std::vector<uint32_t> &cost, uint64_t blocks, std::vector<uint64_t> *items) {
    const uint32_t n = uint32_t(cost.size());
    if (n < 4 * kXcds || blocks == 0 || blocks > 0xFFFFFFFFull) return false;
    std::vector<uint32_t> order(n);
    for (uint32_t q = 0; q < n; ++q) order[q] = q;
    std::stable_sort(order.begin(), order.end(), [&](uint32_t x, uint32_t y) { return cost[x] > cost[y]; });
    std::vector<uint64_t> load(kXcds, 0);
    std::vector<std::vector<uint32_t>> progs(kXcds);
    for (uint32_t q : order) {
        const uint32_t k = uint32_t(std::min_element(load.begin(), load.end()) - load.begin());
        progs[k].push_back(q);
        load[k] += cost[q];
    }
    uint64_t total = 0, top = 0;
    size_t len = 0;
    for (uint32_t k = 0; k < kXcds; ++k) {
        total += load[k];
        top = std::max(top, load[k]);
        len = std::max(len, progs[k].size());
    }
    if (top * 20 * kXcds > total * 21) return false;
    const uint64_t n_wg = uint64_t(len) * blocks * kXcds;
    if (n_wg > 0xFFFFFFFFull) return false;
    items->assign(size_t(n_wg), ~uint64_t(0));
    for (uint32_t k = 0; k < kXcds; ++k) {
        uint64_t i = 0;
        for (uint32_t q : progs[k])
            for (uint64_t bx = 0; bx < blocks; ++bx) (*items)[size_t(k + kXcds * i++)] = uint64_t(q) << 32 | bx;
    }
    return true;
}

ndvm_status many_launch(const ndvm_tape *const *tapes, int n_prog, int64_t L, bool build, ManyLaunch *out) {
    DeviceProps p;
    ndvm_status st = device_props(&p);
    if (st != NDVM_OK) return st;
    const uint32_t S = choose_slots(p, L, n_prog);
    const uint32_t b = reg_budget(p, waves_of(L, n_prog, S), S);
    std::vector<ProgStatic> table(static_cast<size_t>(n_prog), ProgStatic{});
    std::vector<uint64_t> key;
    uint64_t row = 0;
    uint32_t r_launch = 0;
    int n_spill = 0;
    std::vector<uint32_t> cost(static_cast<size_t>(n_prog));
    uint64_t n_mac = 0, n_acc = 0, n_msub = 0, n_block = 0, n_instr = 0;
    std::map<const ndvm_tape *, Schedule> pre;
    if (build && (st = schedule_many(tapes, n_prog, S, b, &pre)) != NDVM_OK) return st;
    for (int q = 0; q < n_prog; ++q) {
        DevProg *dp;
        auto pi = pre.find(tapes[q]);
        Schedule *ps = pi != pre.end() && pi->second.code.size() ? &pi->second : nullptr;
        if ((st = grad_program(const_cast<ndvm_tape *>(tapes[q]), S, b, build, &dp, ps)) != NDVM_OK) return st;
        cost[q] = dp->meta.n_instr;
        uint32_t r_lds = std::min(dp->meta.n_regs, b);
        r_launch = std::max(r_launch, r_lds);
        const bool spills = dp->meta.n_regs > r_lds;
        n_spill += spills;
        out->skips = out->skips || dp->meta.n_skips > 0;
        n_mac += dp->meta.n_mac;
        n_acc += dp->meta.n_acc;
        n_msub += dp->meta.n_msub;
        n_block += dp->meta.n_block;
        n_instr += dp->meta.n_instr;
        table[q] = ProgStatic{dp->code, dp->consts, row, row + dp->meta.n_ckpt_rows + slot::kMaxBlock,
                              dp->meta.hdr_off, r_lds, spills};
        row += ws_rows(*dp, b);
        key.push_back(tapes[q]->id);
        key.push_back((uint64_t(S) << 32) | b);
    }
    out->S = S;
    out->order = dispatch_order(n_mac, n_acc, n_msub, n_block, n_instr);
    out->r_launch = r_launch;
    out->rows = row;
    out->variant = n_spill == 0 ? kLdsOnly : n_spill == n_prog ? kSpill : kPerProgram;
    if (n_prog == 0) return NDVM_OK;
    std::lock_guard<std::mutex> lk(g_table_mu);
    // per-XCD work items (single launches only: at most kMaxProgPerLaunch programs)
    const uint64_t blocks = uint64_t((L + 64 / S - 1) / (64 / S));
    std::vector<uint64_t> ikey = key;
    ikey.push_back(blocks);
    auto ii = g_items.find(ikey);
    if (ii == g_items.end() && build) {
        ItemTable t;
        std::vector<uint64_t> items;
        if (n_prog <= kMaxProgPerLaunch && xcd_items(cost, blocks, &items)) {
            if (hipMalloc(&t.d, items.size() * sizeof(uint64_t)) != hipSuccess) {
                (void)hipGetLastError();
                set_error("hipMalloc of the work-item table failed");
                return NDVM_E_NOMEM;
            }
            if (hipMemcpy(t.d, items.data(), items.size() * sizeof(uint64_t), hipMemcpyHostToDevice) != hipSuccess) {
                (void)hipFree(t.d);
                set_error("copy of the work-item table failed");
                return NDVM_E_DEVICE;
            }
            t.n_wg = uint32_t(items.size());
        }
        ii = g_items.emplace(ikey, t).first;
    }
    if (ii != g_items.end()) {   // a compute call for a lane count never sized keeps the plain grid
        out->d_items = static_cast<const uint64_t *>(ii->second.d);
        out->n_wg = ii->second.n_wg;
    }
    auto it = g_tables.find(key);
    if (it != g_tables.end()) {
        out->d_table = it->second;
        return NDVM_OK;
    }
    if (!build) {
        set_error("no program table for this program set and lane count: size the workspace with "
                  "ndvm_workspace_bytes_many for the same programs and lane count first");
        return NDVM_E_ARG;
    }
    void *d_table = nullptr;
    if (hipMalloc(&d_table, table.size() * sizeof(ProgStatic)) != hipSuccess) {
        (void)hipGetLastError();
        set_error("hipMalloc of the program table failed");
        return NDVM_E_NOMEM;
    }
    if (hipMemcpy(d_table, table.data(), table.size() * sizeof(ProgStatic), hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(d_table);
        set_error("copy of the program table failed");
        return NDVM_E_DEVICE;
    }
    g_tables.emplace(key, d_table);
    out->d_table = d_table;
    return NDVM_OK;
}

template <class F>
ndvm_status guarded(F f) {
    try {
        return f();
    } catch (const std::bad_alloc &) {
        set_error("out of host memory");
        return NDVM_E_NOMEM;
    } catch (const std::exception &e) {
        set_error(std::string("internal error: ") + e.what());
        return NDVM_E_INTERNAL;
    }
}

}  // namespace

extern "C" {

const char *ndvm_last_error(void) { return get_error(); }

ndvm_status ndvm_adam_step(double *params, const double *grad, double *m, double *v, int64_t L, int64_t P,
                           int64_t ld_p, int64_t ld_g, int64_t t, double lr, double beta1, double beta2,
                           double eps, void *stream) {
    return guarded([&]() -> ndvm_status {
        if (L < 0 || P < 0 || ld_p < P || ld_g < P || t < 1 || !(beta1 >= 0.0 && beta1 < 1.0) ||
            !(beta2 >= 0.0 && beta2 < 1.0)) {
            set_error("ndvm_adam_step: bad size, stride, step or beta");
            return NDVM_E_ARG;
        }
        if (L * P == 0) return NDVM_OK;
        if (!params || !grad || !m || !v) {
            set_error("ndvm_adam_step: null buffer");
            return NDVM_E_ARG;
        }
        const AdamArgs a{params, grad, m, v, L, P, ld_p, ld_g, lr, beta1, beta2, eps,
                         1.0 - std::pow(beta1, double(t)), 1.0 - std::pow(beta2, double(t))};
        const hipError_t e = launch_adam(a, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) {
            set_error(std::string("ndvm_adam_step: launch failed: ") + hipGetErrorString(e));
            return NDVM_E_DEVICE;
        }
        return NDVM_OK;
    });
}

void ndvm_free(void *p) { std::free(p); }

ndvm_status ndvm_tape_build(const uint8_t *bytecode, size_t len, uint8_t **tape, size_t *tape_len) {
    return guarded([&]() -> ndvm_status {
        if (!bytecode || !tape || !tape_len) {
            set_error("ndvm_tape_build: null argument");
            return NDVM_E_ARG;
        }
        std::vector<uint8_t> out;
        ndvm_status st = build_tape(bytecode, len, &out);
        if (st != NDVM_OK) return st;
        void *p = std::malloc(out.size());
        if (!p) {
            set_error("out of host memory");
            return NDVM_E_NOMEM;
        }
        std::memcpy(p, out.data(), out.size());
        *tape = static_cast<uint8_t *>(p);
        *tape_len = out.size();
        return NDVM_OK;
    });
}

// Host part of an upload: parse and validate the tape into a new handle.
static ndvm_status new_tape(const uint8_t *bytes, size_t len, int save, bool arms, std::unique_ptr<ndvm_tape> *out) {
    auto h = std::make_unique<ndvm_tape>();
    ndvm_status st = parse_tape(bytes, len, &h->tape);
    if (st != NDVM_OK) return st;
    h->tape_bytes = len;
    h->policy = save;
    h->arms = arms;
    for (const TapeOp &o : h->tape.ops) h->n_selects += o.code == tp::SELECT;
    *out = std::move(h);
    return NDVM_OK;
}

static ndvm_status check_policy(int policy, const char *who) {
    const int save = policy & ~NDVM_BRANCH_SKIP;
    if (save != NDVM_POLICY_RECOMPUTE && save != NDVM_POLICY_SAVE) {
        set_error(std::string(who) + ": unsupported save policy");
        return NDVM_E_UNSUPPORTED;
    }
    return NDVM_OK;
}

ndvm_status ndvm_tape_upload(const uint8_t *bytes, size_t len, int policy, void *stream, ndvm_tape **out) {
    return guarded([&]() -> ndvm_status {
        if (!bytes || !out) {
            set_error("ndvm_tape_upload: null argument");
            return NDVM_E_ARG;
        }
        ndvm_status st = check_policy(policy, "ndvm_tape_upload");
        if (st != NDVM_OK) return st;
        std::unique_ptr<ndvm_tape> h;
        if ((st = new_tape(bytes, len, policy & ~NDVM_BRANCH_SKIP, (policy & NDVM_BRANCH_SKIP) != 0, &h)) != NDVM_OK)
            return st;
        h->id = g_next_id++;
        // schedule the forward program now: scheduling limits surface at upload
        DevProg *fp = nullptr;
        st = fwd_program(h.get(), 4, static_cast<hipStream_t>(stream), &fp);
        if (st != NDVM_OK) return st;
        *out = h.release();
        return NDVM_OK;
    });
}

ndvm_status ndvm_tape_upload_many(const uint8_t *const *tapes, const size_t *lens, int n, int policy, void *stream,
                                  ndvm_tape **out) {
    return guarded([&]() -> ndvm_status {
        if (n < 0 || (n > 0 && (!tapes || !lens || !out))) {
            set_error("ndvm_tape_upload_many: bad argument");
            return NDVM_E_ARG;
        }
        for (int i = 0; i < n; ++i) {
            out[i] = nullptr;
            if (!tapes[i]) {
                set_error("ndvm_tape_upload_many: null tape");
                return NDVM_E_ARG;
            }
        }
        ndvm_status st = check_policy(policy, "ndvm_tape_upload_many");
        if (st != NDVM_OK || n == 0) return st;
        const int save = policy & ~NDVM_BRANCH_SKIP;
        const bool arms = (policy & NDVM_BRANCH_SKIP) != 0;
        // parse and schedule the forward programs on all host threads (the
        // register budget comes from this thread's current device)
        const uint32_t fb = fwd_budget(4);
        std::vector<std::unique_ptr<ndvm_tape>> hs(static_cast<size_t>(n));
        std::vector<Schedule> fw(static_cast<size_t>(n));
        std::vector<ndvm_status> code(static_cast<size_t>(n), NDVM_OK);
        std::vector<std::string> msg(static_cast<size_t>(n));
        std::atomic<int> next{0};
        auto work = [&]() {
            for (int i; (i = next.fetch_add(1)) < n;) {
                try {
                    if ((code[i] = new_tape(tapes[i], lens[i], save, arms, &hs[i])) != NDVM_OK) {
                        msg[i] = get_error();
                        continue;
                    }
                    fw[i] = schedule_forward_of(hs[i].get(), 4, fb);
                } catch (const std::length_error &e) {
                    code[i] = NDVM_E_UNSUPPORTED;
                    msg[i] = std::string("program too large for the device format: ") + e.what();
                } catch (const std::bad_alloc &) {
                    code[i] = NDVM_E_NOMEM;
                    msg[i] = "out of host memory";
                } catch (const std::exception &e) {
                    code[i] = NDVM_E_INTERNAL;
                    msg[i] = std::string("internal error: ") + e.what();
                }
            }
        };
        const int n_threads = std::min(n, int(std::max(1u, std::thread::hardware_concurrency())));
        std::vector<std::thread> pool;
        for (int k = 1; k < n_threads; ++k) pool.emplace_back(work);
        work();
        for (auto &th : pool) th.join();
        for (int i = 0; i < n; ++i)
            if (code[i] != NDVM_OK) {
                set_error("ndvm_tape_upload_many: tape " + std::to_string(i) + ": " + msg[i]);
                return code[i];
            }
        // upload in order; on a failure nothing is returned
        for (int i = 0; i < n; ++i) {
            hs[i]->id = g_next_id++;
            DevProg *fp = nullptr;
            if ((st = fwd_program(hs[i].get(), 4, static_cast<hipStream_t>(stream), &fp, &fw[i])) != NDVM_OK)
                return st;
        }
        for (int i = 0; i < n; ++i) out[i] = hs[i].release();
        return NDVM_OK;
    });
}

ndvm_status ndvm_tape_info_get(const ndvm_tape *t, ndvm_tape_info *out) {
    if (!t || !out) {
        set_error("ndvm_tape_info_get: null argument");
        return NDVM_E_ARG;
    }
    out->n_params = t->tape.n_params;
    out->n_obs = t->tape.n_obs;
    out->n_ops = uint32_t(t->tape.ops.size());
    out->n_consts = uint32_t(t->tape.consts.size());
    out->loss_slot = t->tape.loss;
    out->n_selects = t->n_selects;
    out->tape_bytes = t->tape_bytes;
    return NDVM_OK;
}

void ndvm_tape_free(ndvm_tape *t) {
    if (!t) return;
    {
        std::lock_guard<std::mutex> lk(g_table_mu);
        for (auto it = g_tables.begin(); it != g_tables.end();) {
            bool uses = false;
            for (size_t i = 0; i + 1 < it->first.size(); i += 2) uses = uses || it->first[i] == t->id;
            if (uses) {
                (void)hipFree(it->second);
                it = g_tables.erase(it);
            } else {
                ++it;
            }
        }
        for (auto it = g_items.begin(); it != g_items.end();) {
            bool uses = false;
            for (size_t i = 0; i + 1 < it->first.size(); i += 2) uses = uses || it->first[i] == t->id;
            if (uses) {
                if (it->second.d) (void)hipFree(it->second.d);
                it = g_items.erase(it);
            } else {
                ++it;
            }
        }
    }
    delete t;
}

ndvm_status ndvm_workspace_bytes(const ndvm_tape *tape, int64_t L, int with_grad, size_t *bytes) {
    return guarded([&]() -> ndvm_status {
        if (!tape || !bytes || L < 0) {
            set_error("ndvm_workspace_bytes: bad argument");
            return NDVM_E_ARG;
        }
        DeviceProps p;
        ndvm_status st = device_props(&p);
        if (st != NDVM_OK) return st;
        int64_t Lp = lpad_of(L);
        const uint32_t S = choose_slots(p, L, 1);
        uint64_t rows;
        DevProg *dp;
        if (with_grad) {
            uint32_t b = 0;
            st = single_grad_program(const_cast<ndvm_tape *>(tape), p, L, S, true, &dp, &b);
            if (st != NDVM_OK) return st;
            rows = ws_rows(*dp, b);
        } else {
            uint32_t bf = uint32_t(p.lds_per_block / reg_bytes(S));
            st = fwd_program(const_cast<ndvm_tape *>(tape), S, nullptr, &dp);
            if (st != NDVM_OK) return st;
            rows = ws_rows(*dp, bf);
        }
        *bytes = size_t(rows * uint64_t(Lp) * sizeof(double));
        return NDVM_OK;
    });
}

ndvm_status ndvm_workspace_bytes_many(const ndvm_tape *const *tapes, int n_prog, int64_t L, size_t *bytes) {
    return guarded([&]() -> ndvm_status {
        if (!tapes || n_prog < 0 || !bytes || L < 0) {
            set_error("ndvm_workspace_bytes_many: bad argument");
            return NDVM_E_ARG;
        }
        for (int q = 0; q < n_prog; ++q)
            if (!tapes[q]) {
                set_error("ndvm_workspace_bytes_many: null tape");
                return NDVM_E_ARG;
            }
        ManyLaunch ml;
        ndvm_status st = many_launch(tapes, n_prog, L, true, &ml);
        if (st != NDVM_OK) return st;
        *bytes = size_t(ml.rows * uint64_t(lpad_of(L)) * sizeof(double));
        return NDVM_OK;
    });
}

static ndvm_status check_common(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p,
                                const double *obs, int64_t n_obs, const double *loss, const char *who) {
    if (!tape) {
        set_error(std::string(who) + ": null tape");
        return NDVM_E_ARG;
    }
    if (L < 0 || (L > 0 && (!loss || (tape->tape.n_params > 0 && !params)))) {
        set_error(std::string(who) + ": bad lane count or null buffer");
        return NDVM_E_ARG;
    }
    if (ld_p < int64_t(tape->tape.n_params) || ld_p < 0) {
        set_error(std::string(who) + ": ld_p smaller than the parameter count");
        return NDVM_E_ARG;
    }
    if (n_obs != int64_t(tape->tape.n_obs) || (n_obs > 0 && !obs)) {
        set_error(std::string(who) + ": n_obs does not match the tape");
        return NDVM_E_ARG;
    }
    return NDVM_OK;
}

ndvm_status ndvm_forward(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p, const double *obs,
                         int64_t n_obs, double *loss, void *ws, size_t ws_bytes, void *stream) {
    return guarded([&]() -> ndvm_status {
        ndvm_status st = check_common(tape, params, L, ld_p, obs, n_obs, loss, "ndvm_forward");
        if (st != NDVM_OK) return st;
        if (L == 0) return NDVM_OK;
        DeviceProps p;
        if ((st = device_props(&p)) != NDVM_OK) return st;
        const uint32_t S = choose_slots(p, L, 1);
        DevProg *fp;
        if ((st = fwd_program(const_cast<ndvm_tape *>(tape), S, static_cast<hipStream_t>(stream), &fp)) != NDVM_OK)
            return st;
        const DevProg &dp = *fp;
        uint32_t r_lds = std::min<uint32_t>(dp.meta.n_regs, uint32_t(p.lds_per_block / reg_bytes(S)));
        int64_t Lp = lpad_of(L);
        size_t need = size_t(ws_rows(dp, r_lds) * uint64_t(Lp) * sizeof(double));
        if (need && (!ws || ws_bytes < need)) {
            set_error("ndvm_forward: workspace too small");
            return NDVM_E_NOMEM;
        }
        LaunchArgs A{obs, params, loss, loss, static_cast<double *>(ws), ld_p, 0, L, Lp, 0, 0};
        const bool spills = dp.meta.n_regs > r_lds;
        ProgStatic D{dp.code, dp.consts, 0, uint64_t(dp.meta.n_ckpt_rows) + slot::kMaxBlock, dp.meta.hdr_off, r_lds, spills};
        return check_stream_and_launch(A, nullptr, D, 1, r_lds, spills ? kSpill : kLdsOnly, dp.meta.n_skips > 0,
                                       dispatch_order(dp.meta), S, static_cast<hipStream_t>(stream));
    });
}

// ndvm_grad and its allocation-free variant: `ws` is the caller's workspace
// or the static scratch array's device address.
static ndvm_status grad_impl(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p,
                             const double *obs, int64_t n_obs, double *loss, double *grad, int64_t ld_g, void *ws,
                             size_t ws_bytes, bool static_ws, void *stream, const char *who) {
    ndvm_status st = check_common(tape, params, L, ld_p, obs, n_obs, loss, who);
    if (st != NDVM_OK) return st;
    if (ld_g < int64_t(tape->tape.n_params) || ld_g < 0 || (L > 0 && tape->tape.n_params > 0 && !grad)) {
        set_error(std::string(who) + ": bad grad buffer or ld_g");
        return NDVM_E_ARG;
    }
    if (L == 0) return NDVM_OK;
    DeviceProps p;
    if ((st = device_props(&p)) != NDVM_OK) return st;
    int64_t Lp = lpad_of(L);
    const uint32_t S = choose_slots(p, L, 1);
    uint32_t b = 0;
    DevProg *dp;
    if ((st = single_grad_program(const_cast<ndvm_tape *>(tape), p, L, S, false, &dp, &b)) != NDVM_OK) return st;
    uint32_t r_lds = std::min(dp->meta.n_regs, b);
    size_t need = size_t(ws_rows(*dp, b) * uint64_t(Lp) * sizeof(double));
    if (static_ws) {
        if (need > scratch_bytes()) {
            set_error(std::string(who) + ": this launch needs " + std::to_string(need) +
                      " bytes of workspace, more than the static scratch of " + std::to_string(scratch_bytes()) +
                      " bytes; use ndvm_grad with a caller workspace");
            return NDVM_E_NOMEM;
        }
        const hipError_t e = scratch_address(&ws);
        if (e != hipSuccess) {
            set_error(std::string(who) + ": hipGetSymbolAddress of the scratch array failed: " +
                      hipGetErrorString(e));
            return NDVM_E_DEVICE;
        }
        ws_bytes = scratch_bytes();
    }
    if (need && (!ws || ws_bytes < need)) {
        set_error(std::string(who) + ": workspace too small");
        return NDVM_E_NOMEM;
    }
    double *wsd = static_cast<double *>(ws);
    LaunchArgs A{obs, params, loss, grad, wsd, ld_p, ld_g, L, Lp, 0, 0};
    const bool spills = dp->meta.n_regs > r_lds;
    ProgStatic D{dp->code, dp->consts, 0, uint64_t(dp->meta.n_ckpt_rows) + slot::kMaxBlock, dp->meta.hdr_off, r_lds, spills};
    return check_stream_and_launch(A, nullptr, D, 1, r_lds, spills ? kSpill : kLdsOnly, dp->meta.n_skips > 0,
                                   dispatch_order(dp->meta), S, static_cast<hipStream_t>(stream));
}

ndvm_status ndvm_grad(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p, const double *obs,
                      int64_t n_obs, double *loss, double *grad, int64_t ld_g, void *ws, size_t ws_bytes,
                      void *stream) {
    return guarded([&]() -> ndvm_status {
        return grad_impl(tape, params, L, ld_p, obs, n_obs, loss, grad, ld_g, ws, ws_bytes, false, stream,
                         "ndvm_grad");
    });
}

ndvm_status ndvm_grad_noalloc(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p,
                              const double *obs, int64_t n_obs, double *loss, double *grad, int64_t ld_g,
                              void *stream) {
    return guarded([&]() -> ndvm_status {
        return grad_impl(tape, params, L, ld_p, obs, n_obs, loss, grad, ld_g, nullptr, 0, true, stream,
                         "ndvm_grad_noalloc");
    });
}

// Flattened data axis: L * N lanes.  Workspace: the replay's rows for L*N
// lanes, then the per-point terms [L*N] and term gradients [L*N, P].
static ndvm_status points_layout(const ndvm_tape *tape, int64_t L, int64_t N, bool build, DevProg **dp,
                                 uint32_t *b, uint64_t *replay_bytes, uint64_t *total) {
    DeviceProps p;
    ndvm_status st = device_props(&p);
    if (st != NDVM_OK) return st;
    const int64_t F = L * N;
    const uint32_t S = choose_slots(p, F, 1);
    if ((st = single_grad_program(const_cast<ndvm_tape *>(tape), p, F, S, build, dp, b)) != NDVM_OK) return st;
    *replay_bytes = ws_rows(**dp, *b) * uint64_t(lpad_of(F)) * sizeof(double);
    *total = *replay_bytes + uint64_t(F) * (1 + tape->tape.n_params) * sizeof(double);
    return NDVM_OK;
}

ndvm_status ndvm_workspace_bytes_points(const ndvm_tape *tape, int64_t L, int64_t n_points, size_t *bytes) {
    return guarded([&]() -> ndvm_status {
        if (!tape || !bytes || L < 0 || n_points < 1 || (L > 0 && n_points > INT64_MAX / L)) {
            set_error("ndvm_workspace_bytes_points: bad argument");
            return NDVM_E_ARG;
        }
        DevProg *dp;
        uint32_t b;
        uint64_t rb, total;
        ndvm_status st = points_layout(tape, L, n_points, true, &dp, &b, &rb, &total);
        if (st != NDVM_OK) return st;
        *bytes = size_t(total);
        return NDVM_OK;
    });
}

ndvm_status ndvm_grad_points(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p,
                             const double *points, int64_t n_points, int64_t ld_pt, double scale, double *loss,
                             double *grad, int64_t ld_g, void *ws, size_t ws_bytes, void *stream) {
    return guarded([&]() -> ndvm_status {
        const char *who = "ndvm_grad_points";
        if (!tape) {
            set_error("ndvm_grad_points: null tape");
            return NDVM_E_ARG;
        }
        const int64_t P = tape->tape.n_params, D = tape->tape.n_obs;
        if (L < 0 || n_points < 1 || ld_pt < D || ld_p < P || ld_g < P || (L > 0 && n_points > INT64_MAX / L) ||
            (L > 0 && (!loss || (P > 0 && (!params || !grad)) || (D > 0 && !points)))) {
            set_error(std::string(who) + ": bad lane or point count, stride or null buffer");
            return NDVM_E_ARG;
        }
        if (L == 0) return NDVM_OK;
        DevProg *dp;
        uint32_t b;
        uint64_t rb, total;
        ndvm_status st = points_layout(tape, L, n_points, false, &dp, &b, &rb, &total);
        if (st != NDVM_OK) return st;
        if (!ws || ws_bytes < total) {
            set_error(std::string(who) + ": workspace too small");
            return NDVM_E_NOMEM;
        }
        const int64_t F = L * n_points;
        double *wsd = static_cast<double *>(ws);
        double *term = wsd + rb / sizeof(double), *tgrad = term + F;
        LaunchArgs A{points, params, term, tgrad, wsd, ld_p, P, F, lpad_of(F), 0, 0, n_points, ld_pt};
        const uint32_t r_lds = std::min(dp->meta.n_regs, b);
        const bool spills = dp->meta.n_regs > r_lds;
        ProgStatic D_{dp->code, dp->consts, 0, uint64_t(dp->meta.n_ckpt_rows) + slot::kMaxBlock, dp->meta.hdr_off,
                      r_lds, spills};
        hipStream_t s = static_cast<hipStream_t>(stream);
        DeviceProps pr;
        if ((st = device_props(&pr)) != NDVM_OK) return st;
        st = check_stream_and_launch(A, nullptr, D_, 1, r_lds, spills ? kSpill : kLdsOnly, dp->meta.n_skips > 0,
                                     dispatch_order(dp->meta), choose_slots(pr, F, 1), s);
        if (st != NDVM_OK) return st;
        const hipError_t e = launch_fold_points(term, tgrad, L, n_points, P, scale, loss, grad, ld_g, s);
        if (e != hipSuccess) {
            set_error(std::string(who) + ": fold launch failed: " + hipGetErrorString(e));
            return NDVM_E_DEVICE;
        }
        return NDVM_OK;
    });
}

ndvm_status ndvm_grad_many(const ndvm_tape *const *tapes, int n_prog, const double *params, int64_t L, int64_t ld_p,
                           int64_t prog_stride_p, const double *obs, int64_t n_obs, double *loss, double *grad,
                           int64_t ld_g, int64_t prog_stride_g, void *ws, size_t ws_bytes, void *stream) {
    return guarded([&]() -> ndvm_status {
        if (!tapes || n_prog < 0) {
            set_error("ndvm_grad_many: bad program list");
            return NDVM_E_ARG;
        }
        if (n_prog == 0 || L == 0) return NDVM_OK;
        uint32_t pmax = 0;
        for (int q = 0; q < n_prog; ++q) {
            ndvm_status st = check_common(tapes[q], params, L, ld_p, obs, n_obs, loss, "ndvm_grad_many");
            if (st != NDVM_OK) return st;
            pmax = std::max(pmax, tapes[q]->tape.n_params);
        }
        if (ld_g < int64_t(pmax) || (pmax > 0 && !grad) || prog_stride_p < L * ld_p ||
            prog_stride_g < L * ld_g || L < 0) {
            set_error("ndvm_grad_many: bad strides");
            return NDVM_E_ARG;
        }
        hipStream_t s = static_cast<hipStream_t>(stream);
        const int64_t Lp = lpad_of(L);
        ManyLaunch ml;
        ndvm_status st = many_launch(tapes, n_prog, L, false, &ml);
        if (st != NDVM_OK) return st;
        size_t need = size_t(ml.rows * uint64_t(Lp) * sizeof(double));
        if (need && (!ws || ws_bytes < need)) {
            set_error("ndvm_grad_many: workspace too small");
            return NDVM_E_NOMEM;
        }
        const uint32_t S = ml.S, r_launch = ml.r_launch;
        const int variant = ml.variant;
        void *d_table = ml.d_table;
        ProgStatic none{};
        // programs run on the grid's y axis, at most kMaxProgPerLaunch per launch;
        // later launches see their programs' parameters, outputs and table rows
        // from their first program on (workspace rows are absolute in the table)
        for (int q0 = 0; q0 < n_prog; q0 += kMaxProgPerLaunch) {
            const int nq = std::min(kMaxProgPerLaunch, n_prog - q0);
            LaunchArgs A{obs, params + q0 * prog_stride_p, loss + int64_t(q0) * L,
                         grad ? grad + q0 * prog_stride_g : nullptr, static_cast<double *>(ws), ld_p, ld_g, L, Lp,
                         prog_stride_p, prog_stride_g};
            if (ml.d_items) {   // one launch over every program, laid out per XCD
                A.wg_items = ml.d_items;
                A.n_wg = ml.n_wg;
            }
            st = check_stream_and_launch(A, static_cast<const ProgStatic *>(d_table) + q0, none, uint32_t(nq),
                                         r_launch, variant, ml.skips, ml.order, S, s);
            if (st != NDVM_OK) return st;
        }
        return NDVM_OK;
    });
}

}  // extern "C"
