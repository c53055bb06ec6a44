// Host side of libapml: argument validation, device memory (pool or caller
// allocator), per-phase event timing, and the launch sequence of the forward
// and backward passes (Algorithm 1 of the paper, redesigned as described at
// the top of kernels.hip).
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <unordered_map>
#include <utility>
#include <vector>

#include "../../include/apml.h"
#include "apml_internal.h"

using namespace apml;

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------

namespace {

thread_local std::string g_last_error;

apml_status fail(apml_status st, const std::string &msg)
{
    g_last_error = msg;
    return st;
}

#define HIP_TRY(expr)                                                                          \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail(APML_ERR_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_));   \
    } while (0)

// ---------------------------------------------------------------------------
// device memory: caller allocator or a per-(device, stream) block pool
// ---------------------------------------------------------------------------

struct Memory {
    std::mutex mu;
    apml_alloc_fn user_alloc = nullptr;
    apml_free_fn user_free = nullptr;
    void *user = nullptr;
    // free blocks of the pool, by (device, stream), keyed by block size
    std::map<std::pair<int, hipStream_t>, std::multimap<size_t, void *>> free_blocks;
    std::unordered_map<void *, size_t> block_size; // every block the pool owns
    int64_t in_use = 0, peak = 0, reserved = 0;
    int live_plans = 0;
};

// Mapped pinned host memory for the forward's read-back block, one buffer per
// device, grown on demand; callers hold mu from the launch that writes it to
// the copy that reads it.
struct Pinned {
    std::mutex mu;
    void *host[64] = {};
    void *dev[64] = {};
    size_t bytes[64] = {};
    void *get(int device, size_t n)
    {
        if (device < 0 || device >= 64)
            return nullptr;
        if (bytes[device] < n) {
            if (host[device])
                (void)hipHostFree(host[device]);
            host[device] = dev[device] = nullptr;
            bytes[device] = 0;
            const size_t want = std::max<size_t>(n, 4096);
            if (hipHostMalloc(&host[device], want, hipHostMallocMapped | hipHostMallocPortable) != hipSuccess)
                return host[device] = nullptr;
            if (hipHostGetDevicePointer(&dev[device], host[device], 0) != hipSuccess) {
                (void)hipHostFree(host[device]);
                return host[device] = nullptr;
            }
            bytes[device] = want;
        }
        return host[device];
    }
    void *device_ptr(int device) const { return dev[device]; }
};

Pinned &pinned()
{
    static Pinned *p = new Pinned(); // never destroyed: outlives every plan
    return *p;
}

Memory &mem()
{
    static Memory m;
    return m;
}

size_t round_block(size_t n)
{
    if (n <= (1u << 20))
        return (n + 511) & ~size_t(511);
    return (n + (size_t(1) << 20) - 1) & ~((size_t(1) << 20) - 1);
}

void *pool_alloc(size_t bytes, hipStream_t s, size_t *got)
{
    Memory &m = mem();
    std::lock_guard<std::mutex> lk(m.mu);
    if (m.user_alloc) {
        void *p = m.user_alloc(bytes, (apml_stream)s, m.user);
        if (p) {
            *got = bytes;
            m.in_use += (int64_t)bytes;
            m.peak = std::max(m.peak, m.in_use);
        }
        return p;
    }
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return nullptr;
    const size_t want = round_block(bytes);
    auto &fl = m.free_blocks[{dev, s}];
    auto it = fl.lower_bound(want);
    void *p = nullptr;
    size_t size = want;
    if (it != fl.end() && it->first <= 2 * want + (size_t(1) << 20)) {
        p = it->second;
        size = it->first;
        fl.erase(it);
    } else {
        if (hipMalloc(&p, want) != hipSuccess) {
            // give the cached blocks back and try once more
            (void)hipGetLastError();
            (void)hipDeviceSynchronize();
            for (auto &kv : m.free_blocks)
                for (auto &blk : kv.second) {
                    (void)hipFree(blk.second);
                    m.reserved -= (int64_t)m.block_size[blk.second];
                    m.block_size.erase(blk.second);
                }
            m.free_blocks.clear();
            if (hipMalloc(&p, want) != hipSuccess) {
                (void)hipGetLastError();
                return nullptr;
            }
        }
        m.block_size[p] = want;
        m.reserved += (int64_t)want;
    }
    *got = size;
    m.in_use += (int64_t)size;
    m.peak = std::max(m.peak, m.in_use);
    return p;
}

void pool_free(void *p, size_t size, hipStream_t s)
{
    if (!p)
        return;
    Memory &m = mem();
    std::lock_guard<std::mutex> lk(m.mu);
    m.in_use -= (int64_t)size;
    if (m.user_free) {
        m.user_free(p, size, (apml_stream)s, m.user);
        return;
    }
    int dev = 0;
    (void)hipGetDevice(&dev);
    m.free_blocks[{dev, s}].insert({size, p});
}

// A region that arenas carve from front to back, never giving memory back
// within a call (the static scratch of apml_forward_backward_noalloc).
struct Bump {
    uint8_t *base = nullptr;
    size_t cap = 0;
    size_t used = 0;
    size_t need = 0; // bytes the call asked for when the region ran out
};

// A set of device blocks released together: from the pool (or the caller's
// allocator), or carved from a bump region.
struct Arena {
    hipStream_t stream = nullptr;
    Bump *bump = nullptr;
    std::vector<std::pair<void *, size_t>> blocks;
    int64_t bytes = 0;
    bool failed = false;

    template <typename T> T *get(size_t count)
    {
        if (failed)
            return nullptr;
        const size_t want = std::max<size_t>(count * sizeof(T), 16);
        if (bump) {
            const size_t at = (bump->used + 255) & ~size_t(255);
            if (at > bump->cap || want > bump->cap - at) {
                bump->need = std::max(bump->need, at + want);
                failed = true;
                return nullptr;
            }
            bump->used = at + want;
            bytes += (int64_t)want;
            return reinterpret_cast<T *>(bump->base + at);
        }
        size_t got = 0;
        void *p = pool_alloc(want, stream, &got);
        if (!p) {
            failed = true;
            return nullptr;
        }
        blocks.push_back({p, got});
        bytes += (int64_t)got;
        return static_cast<T *>(p);
    }
    void release()
    {
        for (auto &b : blocks)
            pool_free(b.first, b.second, stream);
        blocks.clear();
        bytes = 0;
    }
    ~Arena() { release(); }
};

// Several arrays cut from one allocation (one pool call instead of one per
// array), each starting on a 256-byte boundary. A first pass with base ==
// nullptr only adds up the size.
struct Carve {
    uint8_t *base = nullptr;
    size_t off = 0;
    template <typename T> T *take(size_t count)
    {
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += (std::max<size_t>(count * sizeof(T), 16) + 255) & ~size_t(255);
        return p;
    }
};

// ---------------------------------------------------------------------------
// per-phase event timing
// ---------------------------------------------------------------------------

const char *kPhaseNames[APML_N_PHASES] = {"stats",    "support", "build",        "softmax",
                                          "sinkhorn", "loss",    "bwd_sinkhorn", "bwd_softmax"};
enum Phase { PH_STATS, PH_SUPPORT, PH_BUILD, PH_SOFTMAX, PH_SINKHORN, PH_LOSS, PH_BWD_SINK, PH_BWD_SOFTMAX };

struct Profiler {
    std::mutex mu;
    bool on = false;
    std::vector<hipEvent_t> spare;
    struct Pending {
        int phase;
        hipEvent_t a, b;
    };
    std::vector<Pending> pending;
    double total[APML_N_PHASES] = {};
    int64_t count[APML_N_PHASES] = {};
};

Profiler &prof()
{
    static Profiler p;
    return p;
}

hipEvent_t take_event()
{
    Profiler &p = prof();
    if (!p.spare.empty()) {
        hipEvent_t e = p.spare.back();
        p.spare.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess)
        return nullptr;
    return e;
}

class PhaseTimer {
  public:
    PhaseTimer(int phase, hipStream_t s, bool enabled = true) : phase_(phase), s_(s)
    {
        if (!enabled)
            return;
        Profiler &p = prof();
        std::lock_guard<std::mutex> lk(p.mu);
        if (!p.on)
            return;
        a_ = take_event();
        b_ = take_event();
        if (a_ && b_)
            (void)hipEventRecord(a_, s_);
    }
    void stop()
    {
        if (!a_ || !b_)
            return;
        (void)hipEventRecord(b_, s_);
        Profiler &p = prof();
        std::lock_guard<std::mutex> lk(p.mu);
        p.pending.push_back({phase_, a_, b_});
        a_ = b_ = nullptr;
    }
    ~PhaseTimer()
    {
        if (a_ || b_) { // abandoned (error path): recycle the events
            Profiler &p = prof();
            std::lock_guard<std::mutex> lk(p.mu);
            if (a_) p.spare.push_back(a_);
            if (b_) p.spare.push_back(b_);
        }
    }

  private:
    int phase_;
    hipStream_t s_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
};

} // namespace

// ---------------------------------------------------------------------------
// the plan
// ---------------------------------------------------------------------------

struct apml_plan {
    int B = 0, N = 0, M = 0, L = 0;
    apml_params prm{};
    Params kp{};
    int device = 0;
    hipStream_t stream = nullptr;
    int64_t stored = 0;     // stored pairs
    int64_t scanned[2] = {0, 0}; // pairs evaluated by the two dense scans
    bool skipping = false;  // the dense scans skipped pairs (large samples)
    int64_t max_sample = 0; // stored pairs of the largest sample
    bool sink_fwd = false;  // per-sample Sinkhorn kernels take this plan (forward)
    bool sink_bwd = false;  // and the reverse sweeps
    bool sink_wide = false; // streamed per-sample Sinkhorn kernels (larger samples)
    bool timed = true;  // phases recorded by the profiler (off for the no-alloc entry point)
    Arena keep;         // everything backward and export need
    DevPlan dv{};       // device arrays (x, y and the backward fields are set per call)
};

namespace {

apml_status validate(const float *x, const float *y, int32_t B, int32_t N, int32_t M, int32_t d,
                     const apml_params &p, const float *loss)
{
    if (!x || !y || !loss)
        return fail(APML_ERR_INVALID_ARG, "x, y and loss must be non-NULL device pointers");
    if (B < 1 || N < 2 || M < 2)
        return fail(APML_ERR_INVALID_ARG, "need B >= 1, N >= 2 and M >= 2 (Eq. 1 needs K > 1)");
    if (d != 3)
        return fail(APML_ERR_UNSUPPORTED, "only d == 3 is supported");
    if ((int64_t)B * N > INT32_MAX / 4 || (int64_t)B * M > INT32_MAX / 4)
        return fail(APML_ERR_UNSUPPORTED, "B*N and B*M must stay below 2^29");
    if (p.struct_size != 0 && p.struct_size < sizeof(apml_params))
        return fail(APML_ERR_INVALID_ARG, "apml_params.struct_size is smaller than this library's struct");
    if (!(p.p_min > 0.0 && p.p_min < 1.0) || !(p.p_min * N > 1.0) || !(p.p_min * M > 1.0))
        return fail(APML_ERR_INVALID_ARG, "need 1/min(N, M) < p_min < 1 (Eq. 1 gives T > 0)");
    if (!(p.tau >= 0.0 && p.tau <= 1.0))
        return fail(APML_ERR_INVALID_ARG, "need 0 <= tau <= 1");
    if (p.n_iter < 0 || p.n_iter > 100000)
        return fail(APML_ERR_INVALID_ARG, "need 0 <= n_iter <= 100000");
    if (!(p.delta >= 0.0) || !(p.eps_gap > 0.0) || !(p.eps_stab >= 0.0) || !(p.eps_dist >= 0.0) ||
        !std::isfinite(p.delta) || !std::isfinite(p.eps_gap) || !std::isfinite(p.eps_stab) ||
        !std::isfinite(p.eps_dist))
        return fail(APML_ERR_INVALID_ARG, "need delta >= 0, eps_gap > 0, eps_stab >= 0, eps_dist >= 0, all finite");
    if (p.dense_scan < APML_SCAN_AUTO || p.dense_scan > APML_SCAN_SKIP)
        return fail(APML_ERR_INVALID_ARG, "dense_scan must be APML_SCAN_AUTO, APML_SCAN_FULL or APML_SCAN_SKIP");
    if (p.gap_mode != APML_GAP_CLAMP && p.gap_mode != APML_GAP_UNIFORM_FALLBACK)
        return fail(APML_ERR_INVALID_ARG, "gap_mode must be APML_GAP_CLAMP or APML_GAP_UNIFORM_FALLBACK");
    if (p.sym_mode != APML_SYM_HALF_SUM && p.sym_mode != APML_SYM_MEAN_DUP)
        return fail(APML_ERR_INVALID_ARG, "sym_mode must be APML_SYM_HALF_SUM or APML_SYM_MEAN_DUP");
    if (p.tgrad_mode != APML_TGRAD_FULL && p.tgrad_mode != APML_TGRAD_DETACHED)
        return fail(APML_ERR_INVALID_ARG, "tgrad_mode must be APML_TGRAD_FULL or APML_TGRAD_DETACHED");
    return APML_OK;
}

// Eq. 1: -log((1 - p) / ((K - 1) p)).
double log_ratio(int K, double p) { return -std::log((1.0 - p) / ((double)(K - 1) * p)); }

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Seconds the forward waits for its read-back before it reports the device
// as stuck: APML_WAIT_TIMEOUT_S if set (0 allowed), else 600.
double wait_deadline_s()
{
    const char *v = std::getenv("APML_WAIT_TIMEOUT_S");
    if (v && *v) {
        char *end = nullptr;
        const double t = std::strtod(v, &end);
        if (end != v && t >= 0.0)
            return t;
    }
    return 600.0;
}

// Waits for the stream by polling: the forward's one synchronisation sits
// on the critical path, and a blocking wait adds the wake-up latency. After
// the first 2 ms the poll sleeps 50 us between queries; past the deadline the
// call fails with APML_ERR_DEVICE instead of waiting for ever.
apml_status wait_for(hipStream_t s)
{
    using clock = std::chrono::steady_clock;
    const auto t0 = clock::now();
    const double deadline = wait_deadline_s();
    for (unsigned n = 0;; ++n) {
        const hipError_t e = hipStreamQuery(s);
        if (e == hipSuccess)
            return APML_OK;
        if (e != hipErrorNotReady)
            return fail(APML_ERR_DEVICE, std::string("hipStreamQuery: ") + hipGetErrorString(e));
        if ((n & 63) != 0)
            continue;
        const double waited = std::chrono::duration<double>(clock::now() - t0).count();
        if (waited > deadline)
            return fail(APML_ERR_DEVICE, "the stream did not reach the forward's read-back within " +
                                             std::to_string(deadline) + " s (APML_WAIT_TIMEOUT_S)");
        if (waited > 2e-3)
            std::this_thread::sleep_for(std::chrono::microseconds(50));
    }
}

// Chunks of the broadcast range so that the support scan has about
// target / 1024 waves per SIMD on 256 CUs, each chunk at least min_chunk
// points long.
void choose_chunks(int B, int n_own, int n_bc, int *S, int *chunk, int min_chunk, int64_t target = 8192)
{
    const int64_t waves = (int64_t)B * ceil_div(n_own, 64);
    int s = (int)std::max<int64_t>(1, (target + waves - 1) / waves);
    s = std::min(s, std::max(1, n_bc / min_chunk));
    int len = ceil_div(n_bc, s);
    len = ceil_div(len, kUnroll) * kUnroll;
    *chunk = len;
    *S = ceil_div(n_bc, len);
}

// The skipping scans pay off when both clouds are large: their sort and
// run selection cost about as much as the full scans of 2048 x 2048 or
// 4096 x 16384 points per sample (measured), and far less than those of two
// clouds of 8192 points or more.
constexpr int kSkipMinPoints = 8192;

bool use_skipping_scans(const apml_params &p, int N, int M)
{
    if (p.dense_scan == APML_SCAN_FULL)
        return false;
    if (p.dense_scan == APML_SCAN_SKIP)
        return true;
    return std::min(N, M) >= kSkipMinPoints;
}

} // namespace

hipError_t apml::set_dynamic_lds(const void *k, size_t bytes)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    static std::mutex mu;
    static std::map<std::pair<int, const void *>, size_t> set; // largest size set per device and kernel
    std::lock_guard<std::mutex> lock(mu);
    const auto key = std::make_pair(dev, k);
    const auto it = set.find(key);
    if (it != set.end() && it->second >= bytes)
        return hipSuccess;
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess)
        set[key] = bytes;
    return e;
}

extern "C" {

void apml_params_default(apml_params *p)
{
    if (!p)
        return;
    p->struct_size = sizeof(apml_params);
    p->n_iter = 10;
    p->p_min = 0.8;
    p->tau = 1e-8;
    p->eps_stab = 1e-8;
    p->delta = 1e-8;
    p->eps_gap = 1e-6;
    p->eps_dist = 1e-12;
    p->dense_scan = APML_SCAN_AUTO;
    p->gap_mode = APML_GAP_CLAMP;
    p->sym_mode = APML_SYM_HALF_SUM;
    p->tgrad_mode = APML_TGRAD_FULL;
}

apml_status apml_plan_destroy(apml_plan *plan)
{
    if (!plan)
        return APML_OK;
    {
        std::lock_guard<std::mutex> lk(mem().mu);
        mem().live_plans--;
    }
    int prev = 0;
    (void)hipGetDevice(&prev);
    if (prev != plan->device)
        (void)hipSetDevice(plan->device);
    plan->keep.release();
    if (prev != plan->device)
        (void)hipSetDevice(prev);
    delete plan;
    return APML_OK;
}

} // extern "C"

namespace {

// Bytes of the read-back block the no-alloc entry point keeps in host memory
// of its own (it bounds B there).
constexpr size_t kStaticReadbackBytes = 64 << 10;

// The forward pass (Alg. 1) into plan, whose device memory comes from
// plan->keep: the pool (or the caller's allocator), or a bump region. The
// arguments are validated.
apml_status run_forward(apml_plan *plan, const float *x, const float *y, int32_t B, int32_t N, int32_t M,
                        const apml_params &prm, float *loss, hipStream_t s)
{
    HIP_TRY(hipGetDevice(&plan->device));
    const int L = prm.n_iter;
    plan->B = B;
    plan->N = N;
    plan->M = M;
    plan->L = L;
    plan->prm = prm;
    plan->stream = s;
    plan->keep.stream = s;
    Params &kp = plan->kp;
    kp.p_min = prm.p_min;
    kp.tau = prm.tau;
    kp.eps_stab = prm.eps_stab;
    kp.delta = prm.delta;
    kp.eps_gap = prm.eps_gap;
    kp.eps_dist = prm.eps_dist;
    kp.log_inv_tau = prm.tau > 0.0 ? -std::log(prm.tau) : HUGE_VAL;
    kp.lk_row = log_ratio(M, prm.p_min);
    kp.lk_col = log_ratio(N, prm.p_min);
    kp.n_iter = L;
    kp.gap_mode = prm.gap_mode;
    kp.sym_mode = prm.sym_mode;
    kp.tgrad_mode = prm.tgrad_mode;

    const int BN = B * N, BM = B * M;
    Arena tmp, dense_tmp; // dense_tmp: scratch of the dense scans, released once the CSR is written
    tmp.stream = s;
    dense_tmp.stream = s;
    tmp.bump = dense_tmp.bump = plan->keep.bump;
    const bool timed = plan->timed;
    Arena &keep = plan->keep;
    DevPlan &dv = plan->dv;
    dv.B = B;
    dv.N = N;
    dv.M = M;
    dv.L = L;
    dv.x = x;
    dv.y = y;
    dv.loss = loss;

    // ---- dense scan 1: minima -------------------------------------------
    // Large samples take the skipping scans over spatially sorted clouds
    // (cull.hip), small ones the full scans (dense.hip).
    const bool skip = use_skipping_scans(prm, N, M);
    plan->skipping = skip;
    dv.m12_row = keep.get<float2>(BN);
    dv.m12_col = keep.get<float2>(BM);
    dv.ctr = keep.get<Counters>(1);
    BuildArgs ba{};
    int32_t *col_cnt = tmp.get<int32_t>(BM); // stored pairs per column, counted by the emission
    ba.col_fill = tmp.get<int32_t>(BM);
    dv.row_ptr = keep.get<int32_t>((size_t)BN + 1);
    dv.col_ptr = keep.get<int32_t>((size_t)BM + 1);
    // full scans
    PairScan ps{};
    EmitArgs ea{};
    // skipping scans
    SpatialArgs sa{};
    CullDir crows{}, ccols{};
    CullEmitArgs ca{};
    int32_t *cnt = nullptr; // stored pairs per row (per (row, chunk) for the full scan)
    int cnt_chunks = 1;
    if (!skip) {
        choose_pair_scan(ps, B, N, M);
        ps.x = x;
        ps.y = y;
        const int owner_blocks = ceil_div(N, kBlock);
        choose_chunks(B, N, M, &ea.S, &ea.chunk, 256);
        // the scratch of both scans in one allocation; the counting pass
        // keeps the first hits of every (row, chunk), at 16-bit offsets
        // within the chunk
        float *E_row = nullptr;
        float4 *ypack = nullptr;
        auto lay = [&](Carve &c) {
            ps.row_partial = c.take<float2>((size_t)ps.S_r * BN);
            ps.col_partial = c.take<float2>((size_t)ps.S_c * BM);
            E_row = c.take<float>(BN);
            ypack = c.take<float4>(BM);
            ea.cnt = c.take<int32_t>((size_t)BN * ea.S);
            if (ea.chunk <= 65536) {
                ea.kst = stage_slots(ea.S);
                ea.stage_narrow = ea.chunk <= 256;
                const size_t staged = (size_t)BN * ea.S * ea.kst;
                ea.stage = c.take<uint16_t>(ea.stage_narrow ? (staged + 1) / 2 : staged);
                const size_t tiles = (size_t)B * ea.S * owner_blocks;
                // a region's base is a 32-bit offset
                ea.spill_cap = std::min<int64_t>((int64_t)tiles * kSpillPerTile, INT32_MAX - kBlock - kTileList);
                ea.spill = c.take<uint16_t>((size_t)ea.spill_cap);
                ea.spill_base = c.take<int32_t>(tiles);
            }
        };
        {
            Carve size;
            lay(size);
            Carve c{dense_tmp.get<uint8_t>(size.off)};
            if (!dense_tmp.failed)
                lay(c);
        }
        if (tmp.failed || dense_tmp.failed || keep.failed)
            return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (statistics)");
        {
            // the statistics phase: the scan and the merge of its partials
            PhaseTimer pt(PH_STATS, s, timed);
            launch_top2_pairs(ps, s);
            HIP_TRY(hipGetLastError());
            FinalizeDir fr{ps.row_partial, x, dv.m12_row, E_row, nullptr, nullptr, nullptr, N, ps.S_r, kp.lk_row};
            FinalizeDir fc{ps.col_partial, y, dv.m12_col, nullptr, ypack, col_cnt, ba.col_fill, M, ps.S_c,
                           kp.lk_col};
            launch_finalize(fr, fc, B, kp, dv.ctr, s); // also clears the counters
            HIP_TRY(hipGetLastError());
            pt.stop();
        }

        // ---- dense scan 2: candidate support -----------------------------
        ea.x = x;
        ea.ypack = ypack;
        ea.E_row = E_row;
        ea.B = B;
        ea.N = N;
        ea.M = M;
        ea.owner_blocks = owner_blocks;
        ea.col_cnt = col_cnt; // cleared by the finalize kernel
        ea.ctr = dv.ctr;
        cnt = ea.cnt;
        cnt_chunks = ea.S;
    } else {
        const int pad_x = pad64(N), pad_y = pad64(M);
        sa.x = x;
        sa.y = y;
        sa.B = B;
        sa.N = N;
        sa.M = M;
        sa.pad_x = pad_x;
        sa.pad_y = pad_y;
        const size_t n_sort = (size_t)B * pad_x + (size_t)B * pad_y;
        sa.ctr = dv.ctr;
        crows.waves = ceil_div(N, kScanRows);
        if (std::max(N, M) > kSortChunkPoints) // chunked sort: the frame from partial boxes
            sa.frame_slices = ceil_div((int64_t)N + M, 16384);
        // the scratch of both scans in one allocation
        Box *batch_x = nullptr, *batch_y = nullptr;
        float *E_row = nullptr;
        float4 *ypack = nullptr;
        auto lay = [&](Carve &c) {
            for (int k = 0; k < 2; ++k) {
                sa.key[k] = c.take<uint32_t>(n_sort);
                sa.val[k] = c.take<uint32_t>(n_sort);
            }
            sa.sx = c.take<float4>((size_t)B * pad_x);
            sa.sy = c.take<float4>((size_t)B * pad_y);
            sa.box_x = c.take<Box>((size_t)B * pad_x / kRun);
            sa.box_y = c.take<Box>((size_t)B * pad_y / kRun);
            sa.frame_part = sa.frame_slices ? c.take<float>((size_t)B * sa.frame_slices * 6) : nullptr;
            batch_x = c.take<Box>((size_t)B * batches(pad_x));
            batch_y = c.take<Box>((size_t)B * batches(pad_y));
            crows.m12s = c.take<float2>((size_t)B * pad_x);
            ccols.m12s = c.take<float2>((size_t)B * pad_y);
            E_row = c.take<float>((size_t)B * pad_x);
            ypack = c.take<float4>((size_t)B * pad_y);
            ca.cnt = c.take<int32_t>(BN);
            ca.stage = c.take<int32_t>((size_t)BN * kCullStage);
            ca.wg_over = c.take<uint8_t>((size_t)B * crows.waves);
        };
        {
            Carve size;
            lay(size);
            Carve c{dense_tmp.get<uint8_t>(size.off)};
            if (!dense_tmp.failed)
                lay(c);
        }
        crows.own = sa.sx;
        crows.bc = sa.sy;
        crows.own_box = sa.box_x;
        crows.bc_box = sa.box_y;
        crows.n_own = N;
        crows.n_bc = M;
        crows.pad_own = pad_x;
        crows.pad_bc = pad_y;
        ccols.own = sa.sy;
        ccols.bc = sa.sx;
        ccols.own_box = sa.box_y;
        ccols.bc_box = sa.box_x;
        ccols.n_own = M;
        ccols.n_bc = N;
        ccols.pad_own = pad_y;
        ccols.pad_bc = pad_x;
        ccols.waves = ceil_div(M, kScanRows);
        crows.bc_batch = batch_y;
        ccols.bc_batch = batch_x;
        if (tmp.failed || dense_tmp.failed || keep.failed)
            return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (statistics)");
        {
            PhaseTimer pt(PH_STATS, s, timed);
            HIP_TRY(launch_spatial_sort(sa, s)); // also clears the counters
            launch_batch_boxes(sa.box_x, sa.box_y, batch_x, batch_y, B, pad_x, pad_y, false, s);
            launch_cull_top2(crows, ccols, B, dv.ctr, s);
            HIP_TRY(hipGetLastError());
            CullFinalizeDir fr{crows.m12s, sa.sx, dv.m12_row, E_row, nullptr, nullptr, nullptr, nullptr, N, pad_x,
                               kp.lk_row};
            CullFinalizeDir fc{ccols.m12s, sa.sy, dv.m12_col, nullptr, ypack, sa.box_y, col_cnt, ba.col_fill, M,
                               pad_y, kp.lk_col};
            launch_cull_finalize(fr, fc, B, kp, s);
            pt.stop();
        }
        // the column batches again, now with their largest emission threshold
        launch_batch_boxes(sa.box_x, sa.box_y, batch_x, batch_y, B, pad_x, pad_y, true, s);
        HIP_TRY(hipGetLastError());

        // ---- dense scan 2: candidate support -----------------------------
        ca.sx = sa.sx;
        ca.E = E_row;
        ca.yp = ypack;
        ca.sy = sa.sy;
        ca.box_x = sa.box_x;
        ca.box_y = sa.box_y;
        ca.batch_y = batch_y;
        ca.B = B;
        ca.N = N;
        ca.M = M;
        ca.pad_x = pad_x;
        ca.pad_y = pad_y;
        ca.waves = crows.waves;
        ca.col_cnt = col_cnt; // cleared by the finalize kernel
        ca.ctr = dv.ctr;
        cnt = ca.cnt;
    }
    int32_t *off_tiles = tmp.get<int32_t>(offsets_scratch_ints(B, N, M));
    // the read-back block: the kernels write it straight into mapped pinned
    // host memory (no copy launch; the buffer is shared, so it is held until
    // copied out), or, with a bump region, into device memory copied out once
    const bool bumped = plan->keep.bump != nullptr;
    uint8_t *rb_dev = bumped ? tmp.get<uint8_t>(readback_bytes(B)) : nullptr;
    if (tmp.failed || dense_tmp.failed)
        return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (support)");
    alignas(16) static thread_local uint8_t rb_static[kStaticReadbackBytes];
    std::vector<uint8_t> rb_vec(bumped ? 0 : readback_bytes(B));
    uint8_t *rb_host = bumped ? rb_static : rb_vec.data();
    std::unique_lock<std::mutex> pin_lock(pinned().mu, std::defer_lock);
    Readback *rb_pin = nullptr;
    if (!bumped) {
        pin_lock.lock();
        rb_pin = (Readback *)pinned().get(plan->device, readback_bytes(B));
        if (!rb_pin)
            return fail(APML_ERR_OUT_OF_MEMORY, "pinned host allocation failed (read-back)");
    }
    Readback *rb = (Readback *)rb_host;
    const int64_t *totals = readback_totals(rb);
    const int32_t *offsets = readback_offsets(rb, B), *pieces = readback_pieces(rb, B);
    {
        PhaseTimer pt(PH_SUPPORT, s, timed);
        if (skip)
            launch_cull_emit_count(ca, s);
        else
            launch_emit_count(ea, s);
        HIP_TRY(hipGetLastError());
        pt.stop();
    }
    // row and column offsets, and what the host needs, in one block
    launch_offsets(cnt, cnt_chunks, col_cnt, dv.ctr, B, N, M, dv.row_ptr, dv.col_ptr, off_tiles,
                   bumped ? (Readback *)rb_dev : (Readback *)pinned().device_ptr(plan->device), s);
    HIP_TRY(hipGetLastError());
    if (bumped)
        HIP_TRY(hipMemcpyAsync(rb_host, rb_dev, readback_bytes(B), hipMemcpyDeviceToHost, s));
    {
        const apml_status ws = wait_for(s);
        if (ws != APML_OK)
            return ws;
    }
    if (!bumped) {
        std::memcpy(rb_host, rb_pin, readback_bytes(B));
        pin_lock.unlock();
    }
    int64_t nnz = 0;
    for (int b = 0; b < B; ++b) {
        if (totals[b] != totals[B + b])
            return fail(APML_ERR_INTERNAL, "row and column counts of the support disagree");
        nnz += totals[b];
    }
    if (nnz > (int64_t)INT32_MAX - 1)
        return fail(APML_ERR_UNSUPPORTED, "more than 2^31 stored pairs: raise tau or lower N*M");
    plan->stored = nnz;
    plan->scanned[0] = skip ? 0 : 2 * (int64_t)B * N * M;
    plan->scanned[1] = skip ? 0 : (int64_t)B * N * M;
    for (int k = 0; skip && k < kScanSlots; ++k) {
        plan->scanned[0] += (int64_t)rb->ctr.scanned[0][k];
        plan->scanned[1] += (int64_t)rb->ctr.scanned[1][k];
    }
    if (offsets[B] != nnz)
        return fail(APML_ERR_INTERNAL, "row offsets disagree with the column counts");
    for (int b = 0; b < B; ++b)
        plan->max_sample = std::max<int64_t>(plan->max_sample, offsets[b + 1] - offsets[b]);
    dv.nnz = nnz;
    const int slots = sinkhorn_slots(N, M, pieces, B);
    plan->sink_fwd = slots > 0;
    plan->sink_bwd = sinkhorn_bwd_fits(slots, plan->max_sample);
    const int wslots = plan->sink_fwd ? 0 : sinkhorn_slots_wide(N, M, pieces, B);
    plan->sink_wide = wslots > 0;

    // ---- sparse structure -------------------------------------------------
    // (with the per-sample Sinkhorn pieces, in one allocation)
    auto lay_pairs = [&](Carve &c) {
        dv.csr_col = c.take<int32_t>(nnz);
        dv.csr_row = c.take<int32_t>(nnz);
        dv.csc_row = c.take<int32_t>(nnz);
        dv.csc_col = c.take<int32_t>(nnz);
        dv.csc_perm = c.take<int32_t>(nnz);
        dv.flags = c.take<uint8_t>(nnz);
        dv.p_row = c.take<float>(nnz);
        dv.p_col = c.take<float>(nnz);
        dv.p0r = c.take<float>(nnz);
        dv.p0c = c.take<float>(nnz);
        dv.cost = c.take<double>(nnz);
        if (plan->sink_fwd) {
            const size_t w = packed_order_words(B, slots);
            for (PackedOrder *pk : {&dv.pk_row, &dv.pk_col}) {
                pk->slots = slots;
                pk->p0 = c.take<float>(w);
                pk->gi = c.take<uint32_t>(w / 2);
                pk->info = c.take<uint32_t>(w / kSinkPiece);
                pk->pos = pk == &dv.pk_col ? c.take<uint32_t>(w / 2) : nullptr;
                pk->n_pos = c.take<int32_t>(B);
            }
        }
        if (plan->sink_wide) {
            const size_t w = packed_order_words(B, wslots);
            for (WideOrder *wk : {&dv.wk_row, &dv.wk_col}) {
                wk->slots = wslots;
                wk->p0 = c.take<float>(w);
                wk->gi = c.take<uint32_t>(w / 2);
                wk->info = c.take<uint32_t>(w / kSinkPiece);
                wk->n_pos = c.take<int32_t>(B);
            }
            dv.split_sync = c.take<uint32_t>((size_t)B * 2 * kSplitSyncStride);
        }
    };
    {
        Carve size;
        lay_pairs(size);
        Carve c{keep.get<uint8_t>(size.off)};
        if (!keep.failed)
            lay_pairs(c);
    }
    // column-major view: per sample in LDS when it fits (with the row
    // softmax), else slots taken by global counters (in the full scan's
    // compaction when no tile is rescanned)
    const char *csc_env = std::getenv("APML_CSC"); // =global: never the per-sample LDS build
    const bool csc_lds = !(csc_env && std::strcmp(csc_env, "global") == 0) && csc_sample_fits(N, M, plan->max_sample);
    const bool placed = !skip && !csc_lds && ea.stage && !rb->ctr.overflow;
    if (!csc_lds) {
        ba.tmp_row = tmp.get<int32_t>(nnz);
        ba.tmp_src = tmp.get<int32_t>(nnz);
    }
    const bool cull_over = skip && rb->ctr.overflow; // a row beyond the staging: written by a second pass
    if (cull_over)
        ca.tmp_col = dense_tmp.get<int32_t>(nnz);
    // pieces of the per-sample Sinkhorn kernels; with staged hits (or the
    // skipping scans) their placement runs in the compaction's (ranking's)
    // launch
    int32_t *place = plan->sink_fwd ? tmp.get<int32_t>((size_t)B * 2 * kSinkOwners) : nullptr;
    int32_t *wplace = plan->sink_wide ? tmp.get<int32_t>((size_t)B * 2 * kSinkOwnersW) : nullptr;
    const bool pieces_placed = place && (skip || (ea.stage && !placed));
    if (tmp.failed || keep.failed || dense_tmp.failed)
        return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (sparse arrays)");
    {
        PhaseTimer pt(PH_BUILD, s, timed);
        if (skip) {
            ca.row_ptr = dv.row_ptr;
            ca.csr_col = dv.csr_col;
            ca.csr_row = dv.csr_row;
            ca.nnz = nnz;
            if (cull_over)
                launch_cull_emit_write(ca, s);
            launch_cull_emit_order(ca, &dv, place, s);
            if (cull_over)
                launch_cull_emit_rank(ca, s);
        } else {
            ea.row_ptr = dv.row_ptr;
            ea.csr_col = dv.csr_col;
            ea.csr_row = dv.csr_row;
            ea.col_ptr = dv.col_ptr;
            ea.col_fill = ba.col_fill;
            ea.tmp_row = ba.tmp_row;
            ea.tmp_src = ba.tmp_src;
            ea.csc_col = dv.csc_col;
            if (ea.stage)
                launch_emit_compact(ea, rb->ctr.overflow != 0, placed, &dv, pieces_placed ? place : nullptr, s);
            else
                launch_emit_write(ea, s);
        }
        if (csc_lds) {
            // built with the row softmax below
        } else if (placed) {
            launch_csc_sort(dv, ba, s);
        } else {
            launch_csc_build(dv, ba, s);
        }
        HIP_TRY(hipGetLastError());
        pt.stop();
    }
    dense_tmp.release();

    // ---- temperatures, softmaxes, P0 ---------------------------------------
    // the per-point arrays of the plan (one allocation, taken once the
    // scans' scratch is released, so that the two never coexist)
    {
        auto lay = [&](Carve &c) {
            dv.T_row = c.take<double>(BN);
            dv.C1_row = c.take<double>(BN);
            dv.g_row = c.take<double>(BN);
            dv.T_col = c.take<double>(BM);
            dv.C1_col = c.take<double>(BM);
            dv.g_col = c.take<double>(BM);
            dv.pos_row = c.take<int32_t>(2 * (size_t)BN);
            dv.pos_col = c.take<int32_t>(2 * (size_t)BM);
            dv.clamp_row = c.take<uint8_t>(BN);
            dv.clamp_col = c.take<uint8_t>(BM);
            // (+ kSinkOwnersW: the split kernels read a sample's vector in
            // whole chunks of lanes, past its end)
            dv.alpha = c.take<double>((size_t)(L + 1) * BN + kSinkOwnersW);
            dv.beta = c.take<double>((size_t)(L + 1) * BM + kSinkOwnersW);
            dv.dvec = c.take<double>(BN);
        };
        Carve size;
        lay(size);
        Carve c{keep.get<uint8_t>(size.off)};
        if (keep.failed)
            return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (plan)");
        lay(c);
    }
    // the per-sample Sinkhorn path: the column softmax writes each pair into
    // its pieces (no separate packing launch)
    if (plan->sink_fwd) {
        if (!pieces_placed)
            launch_place(dv, place, s);
        dv.sink_place = place;
    }
    {
        PhaseTimer pt(PH_SOFTMAX, s, timed);
        if (csc_lds) {
            HIP_TRY(launch_csc_and_softmax(dv, kp, plan->max_sample, s));
        } else {
            launch_softmax(dv, kp, s);
            HIP_TRY(hipGetLastError());
        }
        pt.stop();
    }

    // ---- Sinkhorn (Eq. 3, Eq. 4) and the loss ------------------------------
    {
        PhaseTimer pt(PH_SINKHORN, s, timed);
        if (plan->sink_fwd) {
            dv.sink_place = nullptr; // scratch of this call
            HIP_TRY(launch_sinkhorn_fwd(dv, prm.eps_stab, s));
        } else if (plan->sink_wide) {
            launch_wide_pack(dv, wplace, s);
            HIP_TRY(launch_sinkhorn_fwd_wide(dv, prm.eps_stab, s));
        } else {
            launch_sinkhorn_fwd_steps(dv, prm.eps_stab, s);
            HIP_TRY(hipGetLastError());
        }
        pt.stop();
    }
    tmp.release();
    return APML_OK;
}

} // namespace

extern "C" {

apml_status apml_forward(const float *x, const float *y, int32_t B, int32_t N, int32_t M,
                         int32_t d, const apml_params *params, float *loss, apml_plan **plan_out,
                         apml_stream stream)
{
    g_last_error.clear();
    if (plan_out)
        *plan_out = nullptr;
    apml_params prm;
    apml_params_default(&prm);
    if (params)
        prm = *params;
    apml_status st = validate(x, y, B, N, M, d, prm, loss);
    if (st != APML_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;

    apml_plan *plan = new apml_plan();
    {
        std::lock_guard<std::mutex> lk(mem().mu);
        mem().live_plans++;
    }
    struct Guard {
        apml_plan *p;
        ~Guard() { apml_plan_destroy(p); }
    } guard{plan};
    st = run_forward(plan, x, y, B, N, M, prm, loss, s);
    if (st != APML_OK)
        return st;
    if (plan_out) {
        guard.p = nullptr;
        *plan_out = plan;
    }
    return APML_OK;
}

} // extern "C"

namespace {

// The backward pass (Sec. III-D) of a plan; scratch from the pool or from the
// plan's bump region.
apml_status run_backward(apml_plan *plan, const float *x, const float *y, const float *grad_loss,
                         float *grad_x, float *grad_y, hipStream_t s)
{
    Arena tmp;
    tmp.stream = s;
    tmp.bump = plan->keep.bump;
    DevPlan dv = plan->dv;
    dv.x = x;
    dv.y = y;
    dv.grad_loss = grad_loss;
    dv.grad_x = grad_x;
    dv.grad_y = grad_y;
    dv.yr = dv.yc = nullptr;
    // the split streamed reverse kernel exchanges the owners' factors in memory
    const bool split = dv.L > 0 && plan->sink_wide && sinkhorn_split_factor(plan->B) > 1;
    // On the per-iteration path the row-order sweep adjoint becomes the final
    // adjoint in place (k_bwd_final reads and writes the same pair), and the
    // cost adjoint reuses the column-order copy, dead once the sweeps end.
    auto lay = [&](Carve &c) {
        dv.adj = c.take<double>(plan->stored);
        if (dv.L > 0 && plan->sink_wide) {
            const size_t w = packed_order_words(plan->B, dv.wk_row.slots);
            dv.wr = c.take<float>(w);
            dv.wc = c.take<float>(w);
            dv.cbar = c.take<double>(plan->stored);
            if (split) {
                // one region per phase, each padded by kSinkOwnersW words
                dv.yr = c.take<float>((size_t)dv.L * ((size_t)plan->B * plan->N + kSinkOwnersW));
                dv.yc = c.take<float>((size_t)dv.L * ((size_t)plan->B * plan->M + kSinkOwnersW));
            }
        } else if (dv.L > 0 && !plan->sink_bwd) {
            dv.rz = dv.adj;
            dv.kz = c.take<double>(plan->stored);
            dv.cbar = dv.kz;
            dv.xyr = c.take<double4>((size_t)plan->B * plan->N);
            dv.xyc = c.take<double4>((size_t)plan->B * plan->M);
        } else {
            dv.cbar = c.take<double>(plan->stored);
        }
    };
    {
        Carve size;
        lay(size);
        Carve c{tmp.get<uint8_t>(size.off)};
        if (!tmp.failed)
            lay(c);
    }
    if (tmp.failed)
        return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (backward)");
    {
        PhaseTimer pt(PH_BWD_SINK, s, plan->timed);
        if (dv.L > 0) {
            if (plan->sink_bwd) {
                HIP_TRY(launch_sinkhorn_bwd(dv, plan->max_sample, s));
            } else if (plan->sink_wide) {
                HIP_TRY(launch_sinkhorn_bwd_wide(dv, s));
            } else {
                launch_sinkhorn_bwd_steps(dv, s);
                HIP_TRY(hipGetLastError());
            }
        }
        pt.stop();
    }
    {
        PhaseTimer pt(PH_BWD_SOFTMAX, s, plan->timed);
        // double-precision P where the reverse sweeps keep the adjoint in
        // double too (per-iteration sweeps), or where there are none
        const bool double_p = dv.L == 0 || (!plan->sink_bwd && !plan->sink_wide);
        launch_bwd_softmax(dv, plan->kp, double_p, s);
        HIP_TRY(hipGetLastError());
        pt.stop();
    }
    tmp.release();
    return APML_OK;
}

} // namespace

extern "C" {

apml_status apml_backward(apml_plan *plan, const float *x, const float *y, const float *grad_loss,
                          float *grad_x, float *grad_y, apml_stream stream)
{
    g_last_error.clear();
    if (!plan || !x || !y || !grad_loss || !grad_x)
        return fail(APML_ERR_INVALID_ARG, "plan, x, y, grad_loss and grad_x must be non-NULL");
    return run_backward(plan, x, y, grad_loss, grad_x, grad_y, (hipStream_t)stream);
}

} // extern "C"

// ---------------------------------------------------------------------------
// forward + backward without allocation
// ---------------------------------------------------------------------------

// Device scratch of apml_forward_backward_noalloc: every array of the plan and
// every temporary of one forward + backward call is carved from it, front to
// back. Each device the library runs on holds its own copy until the process
// ends. Host code never uses this name as an address: the kernels receive the
// per-device address that hipGetSymbolAddress returns.
static __device__ __align__(256) unsigned char scratch[APML_NOALLOC_SCRATCH_BYTES];

namespace {

struct ScratchAddresses {
    std::mutex mu;
    void *ptr[64] = {};
};

ScratchAddresses &scratch_addresses()
{
    static ScratchAddresses *a = new ScratchAddresses(); // never destroyed
    return *a;
}

// The device address of the scratch array on the current device, looked up
// once per device (with that device current).
apml_status scratch_of_current_device(void **out)
{
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= 64)
        return fail(APML_ERR_UNSUPPORTED, "device index beyond 63");
    ScratchAddresses &a = scratch_addresses();
    std::lock_guard<std::mutex> lk(a.mu);
    if (!a.ptr[dev]) {
        void *p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p)
            return fail(APML_ERR_DEVICE, "hipGetSymbolAddress returned NULL for the static scratch");
        a.ptr[dev] = p;
    }
    *out = a.ptr[dev];
    return APML_OK;
}

std::string mib(size_t bytes)
{
    char buf[32];
    std::snprintf(buf, sizeof buf, "%.1f MiB", (double)bytes / (1 << 20));
    return buf;
}

} // namespace

extern "C" {

apml_status apml_forward_backward_noalloc(const float *x, const float *y, int32_t B, int32_t N, int32_t M,
                                          int32_t d, const apml_params *params, float *loss,
                                          const float *grad_loss, float *grad_x, float *grad_y,
                                          apml_stream stream)
{
    g_last_error.clear();
    apml_params prm;
    apml_params_default(&prm);
    if (params)
        prm = *params;
    apml_status st = validate(x, y, B, N, M, d, prm, loss);
    if (st != APML_OK)
        return st;
    if (grad_x && !grad_loss)
        return fail(APML_ERR_INVALID_ARG, "grad_loss must be non-NULL when grad_x is");
    if (readback_bytes(B) > kStaticReadbackBytes)
        return fail(APML_ERR_UNSUPPORTED, "B is too large for apml_forward_backward_noalloc (at most " +
                                              std::to_string((kStaticReadbackBytes - sizeof(Readback) - 4) / 36) +
                                              " samples)");
    void *base = nullptr;
    st = scratch_of_current_device(&base);
    if (st != APML_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    Bump bump;
    bump.base = static_cast<uint8_t *>(base);
    bump.cap = APML_NOALLOC_SCRATCH_BYTES;
    apml_plan plan; // host state on the stack; its arrays live in the scratch
    plan.timed = false;
    plan.keep.bump = &bump;
    plan.keep.stream = s;
    auto too_large = [&](apml_status r) {
        if (r == APML_ERR_OUT_OF_MEMORY && bump.need > bump.cap)
            return fail(APML_ERR_OUT_OF_MEMORY, "the call needs " + mib(bump.need) +
                                                    " of device scratch; apml_forward_backward_noalloc has " +
                                                    mib(bump.cap) + " (APML_NOALLOC_SCRATCH_BYTES)");
        return r;
    };
    st = run_forward(&plan, x, y, B, N, M, prm, loss, s);
    if (st != APML_OK)
        return too_large(st);
    if (grad_x) {
        st = run_backward(&plan, x, y, grad_loss, grad_x, grad_y, s);
        if (st != APML_OK)
            return too_large(st);
    }
    return APML_OK;
}

} // extern "C"

// ---------------------------------------------------------------------------
// dense APML
// ---------------------------------------------------------------------------

struct apml_dense_plan {
    int B = 0, N = 0, M = 0, d = 0, L = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    Arena keep; // the per-owner vectors, P0, the plan, the Sinkhorn sums
    DenseDev dv{};
};

namespace {

apml_status validate_dense(const float *x, const float *y, int32_t B, int32_t N, int32_t M, int32_t d,
                           const apml_params &p, const float *loss)
{
    if (!x || !y || !loss)
        return fail(APML_ERR_INVALID_ARG, "x, y and loss must be non-NULL device pointers");
    if (B < 1 || N < 2 || M < 2)
        return fail(APML_ERR_INVALID_ARG, "need B >= 1, N >= 2 and M >= 2 (Eq. 1 needs K > 1)");
    if (d < 1 || d > kDenseMaxD)
        return fail(APML_ERR_UNSUPPORTED, "the dense path takes 1 <= d <= " + std::to_string(kDenseMaxD));
    if ((int64_t)B * N > INT32_MAX / 4 || (int64_t)B * M > INT32_MAX / 4)
        return fail(APML_ERR_UNSUPPORTED, "B*N and B*M must stay below 2^29");
    if ((int64_t)B * N * M > ((int64_t)1 << 40))
        return fail(APML_ERR_UNSUPPORTED, "B*N*M beyond 2^40 pairs");
    if (p.struct_size != 0 && p.struct_size < sizeof(apml_params))
        return fail(APML_ERR_INVALID_ARG, "apml_params.struct_size is smaller than this library's struct");
    if (!(p.p_min > 0.0 && p.p_min < 1.0) || !(p.p_min * N > 1.0) || !(p.p_min * M > 1.0))
        return fail(APML_ERR_INVALID_ARG, "need 1/min(N, M) < p_min < 1 (Eq. 1 gives T > 0)");
    if (p.n_iter < 0 || p.n_iter > 100000)
        return fail(APML_ERR_INVALID_ARG, "need 0 <= n_iter <= 100000");
    if (!(p.delta >= 0.0) || !(p.eps_gap > 0.0) || !(p.eps_stab >= 0.0) || !(p.eps_dist >= 0.0) ||
        !std::isfinite(p.delta) || !std::isfinite(p.eps_gap) || !std::isfinite(p.eps_stab) ||
        !std::isfinite(p.eps_dist))
        return fail(APML_ERR_INVALID_ARG, "need delta >= 0, eps_gap > 0, eps_stab >= 0, eps_dist >= 0, all finite");
    if (p.gap_mode != APML_GAP_CLAMP || p.sym_mode != APML_SYM_HALF_SUM)
        return fail(APML_ERR_UNSUPPORTED, "the dense path takes the clamp and the half sum only");
    if (p.tgrad_mode != APML_TGRAD_FULL && p.tgrad_mode != APML_TGRAD_DETACHED)
        return fail(APML_ERR_INVALID_ARG, "tgrad_mode must be APML_TGRAD_FULL or APML_TGRAD_DETACHED");
    return APML_OK;
}

// Per-owner vectors of one direction, carved from c.
void lay_side(Carve &c, DenseSide &s, size_t n)
{
    s.k1 = c.take<int32_t>(n);
    s.k2 = c.take<int32_t>(n);
    s.c1 = c.take<double>(n);
    s.g = c.take<double>(n);
    s.T = c.take<double>(n);
    s.Z = c.take<double>(n);
    s.clamped = c.take<uint8_t>(n);
    s.sigma = c.take<double>(n);
    s.gbar = c.take<double>(n);
    s.e = c.take<double>(n);
}

} // namespace

extern "C" {

apml_status apml_dense_plan_destroy(apml_dense_plan *plan)
{
    if (!plan)
        return APML_OK;
    {
        std::lock_guard<std::mutex> lk(mem().mu);
        mem().live_plans--;
    }
    int prev = 0;
    (void)hipGetDevice(&prev);
    if (prev != plan->device)
        (void)hipSetDevice(plan->device);
    plan->keep.release();
    if (prev != plan->device)
        (void)hipSetDevice(prev);
    delete plan;
    return APML_OK;
}

apml_status apml_dense_forward(const float *x, const float *y, int32_t B, int32_t N, int32_t M, int32_t d,
                               const apml_params *params, float *loss, apml_dense_plan **plan_out,
                               apml_stream stream)
{
    g_last_error.clear();
    if (plan_out)
        *plan_out = nullptr;
    apml_params prm;
    apml_params_default(&prm);
    if (params)
        prm = *params;
    apml_status st = validate_dense(x, y, B, N, M, d, prm, loss);
    if (st != APML_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    apml_dense_plan *plan = new apml_dense_plan();
    {
        std::lock_guard<std::mutex> lk(mem().mu);
        mem().live_plans++;
    }
    struct Guard {
        apml_dense_plan *p;
        ~Guard() { apml_dense_plan_destroy(p); }
    } guard{plan};
    HIP_TRY(hipGetDevice(&plan->device));
    plan->B = B;
    plan->N = N;
    plan->M = M;
    plan->d = d;
    plan->L = prm.n_iter;
    plan->stream = s;
    plan->keep.stream = s;
    DenseDev &D = plan->dv;
    D.B = B;
    D.N = N;
    D.M = M;
    D.d = d;
    D.L = prm.n_iter;
    D.delta = prm.delta;
    D.eps_gap = prm.eps_gap;
    D.eps_stab = prm.eps_stab;
    D.eps_dist = prm.eps_dist;
    D.tgrad_full = prm.tgrad_mode == APML_TGRAD_FULL;
    D.x = x;
    D.y = y;
    D.loss = loss;
    dense_chunks(B, N, M, &D.chunks, &D.chunk);
    const size_t BN = (size_t)B * N, BM = (size_t)B * M, pairs = (size_t)B * N * M, L = (size_t)prm.n_iter;
    auto lay = [&](Carve &c) {
        lay_side(c, D.row, BN);
        lay_side(c, D.col, BM);
        D.S = c.take<double>(std::max<size_t>(L, 1) * BM);
        D.R = c.take<double>(std::max<size_t>(L, 1) * BN);
        D.a_cum = c.take<double>((L + 1) * BN);
        D.c_cum = c.take<double>((L + 1) * BM);
        D.P0 = c.take<float>(pairs);
        D.P = c.take<float>(pairs);
    };
    {
        Carve size;
        lay(size);
        Carve c{plan->keep.get<uint8_t>(size.off)};
        if (plan->keep.failed)
            return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (dense plan)");
        lay(c);
    }
    Arena tmp;
    tmp.stream = s;
    D.part = tmp.get<double>((size_t)D.chunks * BM);
    if (tmp.failed)
        return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (dense scratch)");
    launch_dense_forward(D, log_ratio(M, prm.p_min), log_ratio(N, prm.p_min), s);
    HIP_TRY(hipGetLastError());
    D.part = nullptr;
    tmp.release();
    if (plan_out) {
        guard.p = nullptr;
        *plan_out = plan;
    }
    return APML_OK;
}

apml_status apml_dense_backward(apml_dense_plan *plan, const float *x, const float *y, const float *grad_loss,
                                float *grad_x, float *grad_y, apml_stream stream)
{
    g_last_error.clear();
    if (!plan || !x || !y || !grad_loss || !grad_x)
        return fail(APML_ERR_INVALID_ARG, "plan, x, y, grad_loss and grad_x must be non-NULL");
    hipStream_t s = (hipStream_t)stream;
    DenseDev D = plan->dv;
    D.x = x;
    D.y = y;
    D.grad_loss = grad_loss;
    D.grad_x = grad_x;
    D.grad_y = grad_y;
    const size_t BM = (size_t)plan->B * plan->M, pairs = (size_t)plan->B * plan->N * plan->M;
    Arena tmp;
    tmp.stream = s;
    D.A = tmp.get<double>(pairs);
    D.part = tmp.get<double>((size_t)D.chunks * BM * (size_t)plan->d);
    if (tmp.failed)
        return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed (dense backward)");
    launch_dense_backward(D, s);
    HIP_TRY(hipGetLastError());
    tmp.release();
    return APML_OK;
}

apml_status apml_plan_get_info(const apml_plan *plan, apml_plan_info *info)
{
    if (!plan || !info)
        return fail(APML_ERR_INVALID_ARG, "plan and info must be non-NULL");
    info->B = plan->B;
    info->N = plan->N;
    info->M = plan->M;
    info->n_iter = plan->L;
    info->stored_pairs = plan->stored;
    info->bytes = plan->keep.bytes;
    info->scanned_min = plan->scanned[0];
    info->scanned_support = plan->scanned[1];
    return APML_OK;
}

apml_status apml_plan_nnz(const apml_plan *plan, int64_t *nnz)
{
    if (!plan || !nnz)
        return fail(APML_ERR_INVALID_ARG, "plan and nnz must be non-NULL");
    hipStream_t s = plan->stream;
    Arena tmp;
    tmp.stream = s;
    const int chunks = count_support_chunks(plan->max_sample);
    const size_t parts = (size_t)plan->B * chunks;
    unsigned long long *d = tmp.get<unsigned long long>(parts);
    if (tmp.failed)
        return fail(APML_ERR_OUT_OF_MEMORY, "device allocation failed");
    launch_count_support(plan->dv.row_ptr, plan->dv.flags, plan->B, plan->N, chunks, d, s);
    HIP_TRY(hipGetLastError());
    std::vector<unsigned long long> h(parts);
    Counters hc{};
    HIP_TRY(hipMemcpyAsync(h.data(), d, sizeof(unsigned long long) * parts, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(&hc, plan->dv.ctr, sizeof(Counters), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    for (int b = 0; b < plan->B; ++b) {
        int64_t n = 0;
        for (int c = 0; c < chunks; ++c)
            n += (int64_t)h[(size_t)b * chunks + c];
        nnz[b] = n;
    }
    if (hc.error & 3u)
        return fail(APML_ERR_INTERNAL, "a row or column minimum was not found among its stored pairs");
    if (hc.error & 4u)
        return fail(APML_ERR_DEVICE, "the workgroups sharing a sample in the split Sinkhorn kernels did not all "
                                     "arrive at a meeting (bounded wait expired)");
    return APML_OK;
}

} // extern "C"

namespace {

template <typename T>
apml_status copy_range(std::vector<T> &dst, const T *src, int64_t begin, int64_t count, hipStream_t s)
{
    dst.resize((size_t)std::max<int64_t>(count, 0));
    if (count > 0)
        HIP_TRY(hipMemcpyAsync(dst.data(), src + begin, sizeof(T) * count, hipMemcpyDeviceToHost, s));
    return APML_OK;
}

#define TRY(expr)                                                                              \
    do {                                                                                       \
        apml_status st_ = (expr);                                                              \
        if (st_ != APML_OK)                                                                    \
            return st_;                                                                        \
    } while (0)

} // namespace

extern "C" {

apml_status apml_plan_export(const apml_plan *plan, int32_t b, int64_t capacity, int32_t *oi,
                             int32_t *oj, uint8_t *oflags, float *op_row, float *op_col, float *op0,
                             float *ov)
{
    if (!plan)
        return fail(APML_ERR_INVALID_ARG, "plan must be non-NULL");
    if (b < 0 || b >= plan->B)
        return fail(APML_ERR_INVALID_ARG, "sample index out of range");
    const int N = plan->N, M = plan->M, L = plan->L;
    hipStream_t s = plan->stream;
    std::vector<int32_t> rp, cp;
    TRY(copy_range(rp, plan->dv.row_ptr, (int64_t)b * N, N + 1, s));
    TRY(copy_range(cp, plan->dv.col_ptr, (int64_t)b * M, M + 1, s));
    HIP_TRY(hipStreamSynchronize(s));
    const int64_t t0 = rp[0], t1 = rp[N], q0 = cp[0], q1 = cp[M];
    std::vector<int32_t> col, perm;
    std::vector<uint8_t> fl;
    std::vector<float> prow, pcol, p0;
    std::vector<double> al, be;
    TRY(copy_range(col, plan->dv.csr_col, t0, t1 - t0, s));
    TRY(copy_range(fl, plan->dv.flags, t0, t1 - t0, s));
    TRY(copy_range(prow, plan->dv.p_row, t0, t1 - t0, s));
    TRY(copy_range(p0, plan->dv.p0r, t0, t1 - t0, s));
    TRY(copy_range(perm, plan->dv.csc_perm, q0, q1 - q0, s));
    TRY(copy_range(pcol, plan->dv.p_col, q0, q1 - q0, s));
    const size_t BN = (size_t)plan->B * N, BM = (size_t)plan->B * M;
    TRY(copy_range(al, plan->dv.alpha, (int64_t)(L * BN + (size_t)b * N), N, s));
    TRY(copy_range(be, plan->dv.beta, (int64_t)(L * BM + (size_t)b * M), M, s));
    HIP_TRY(hipStreamSynchronize(s));
    std::vector<float> pcol_rm(t1 - t0, 0.0f);
    for (int64_t q = 0; q < q1 - q0; ++q)
        pcol_rm[perm[q] - t0] = pcol[q];
    int64_t n = 0;
    for (int i = 0; i < N; ++i)
        for (int64_t t = rp[i]; t < rp[i + 1]; ++t) {
            const int64_t k = t - t0;
            if (!fl[k])
                continue;
            if (n >= capacity)
                return fail(APML_ERR_INVALID_ARG, "capacity is smaller than the sample's support");
            const int j = col[k];
            if (oi) oi[n] = i;
            if (oj) oj[n] = j;
            if (oflags) oflags[n] = fl[k];
            if (op_row) op_row[n] = prow[k];
            if (op_col) op_col[n] = pcol_rm[k];
            if (op0) op0[n] = p0[k];
            if (ov) ov[n] = (float)(al[i] * (double)p0[k] * be[j]);
            ++n;
        }
    return APML_OK;
}

apml_status apml_plan_export_stats(const apml_plan *plan, int32_t b, double *T_row, int32_t *j1,
                                   int32_t *j2, uint8_t *row_clamped, double *T_col, int32_t *i1,
                                   int32_t *i2, uint8_t *col_clamped)
{
    if (!plan)
        return fail(APML_ERR_INVALID_ARG, "plan must be non-NULL");
    if (b < 0 || b >= plan->B)
        return fail(APML_ERR_INVALID_ARG, "sample index out of range");
    const int N = plan->N, M = plan->M;
    hipStream_t s = plan->stream;
    std::vector<double> tr, tc;
    std::vector<int32_t> pr, pc, col, row;
    std::vector<uint8_t> cr, cc;
    TRY(copy_range(tr, plan->dv.T_row, (int64_t)b * N, N, s));
    TRY(copy_range(tc, plan->dv.T_col, (int64_t)b * M, M, s));
    TRY(copy_range(pr, plan->dv.pos_row, 2 * (int64_t)b * N, 2 * (int64_t)N, s));
    TRY(copy_range(pc, plan->dv.pos_col, 2 * (int64_t)b * M, 2 * (int64_t)M, s));
    TRY(copy_range(cr, plan->dv.clamp_row, (int64_t)b * N, N, s));
    TRY(copy_range(cc, plan->dv.clamp_col, (int64_t)b * M, M, s));
    TRY(copy_range(col, plan->dv.csr_col, 0, plan->stored, s));
    TRY(copy_range(row, plan->dv.csc_row, 0, plan->stored, s));
    HIP_TRY(hipStreamSynchronize(s));
    auto at = [](const std::vector<int32_t> &v, int32_t k) { return k >= 0 && (size_t)k < v.size() ? v[k] : -1; };
    for (int i = 0; i < N; ++i) {
        if (T_row) T_row[i] = tr[i];
        if (j1) j1[i] = at(col, pr[2 * i]);
        if (j2) j2[i] = at(col, pr[2 * i + 1]);
        if (row_clamped) row_clamped[i] = cr[i];
    }
    for (int j = 0; j < M; ++j) {
        if (T_col) T_col[j] = tc[j];
        if (i1) i1[j] = at(row, pc[2 * j]);
        if (i2) i2[j] = at(row, pc[2 * j + 1]);
        if (col_clamped) col_clamped[j] = cc[j];
    }
    return APML_OK;
}

apml_status apml_set_allocator(apml_alloc_fn alloc, apml_free_fn free_fn, void *user)
{
    if ((alloc == nullptr) != (free_fn == nullptr))
        return fail(APML_ERR_INVALID_ARG, "alloc and free must both be set or both be NULL");
    Memory &m = mem();
    std::lock_guard<std::mutex> lk(m.mu);
    if (m.live_plans > 0)
        return fail(APML_ERR_INVALID_ARG, "cannot change the allocator while plans are alive");
    m.user_alloc = alloc;
    m.user_free = free_fn;
    m.user = user;
    return APML_OK;
}

apml_status apml_get_memory_stats(apml_memory_stats *stats)
{
    if (!stats)
        return fail(APML_ERR_INVALID_ARG, "stats must be non-NULL");
    Memory &m = mem();
    std::lock_guard<std::mutex> lk(m.mu);
    stats->in_use = m.in_use;
    stats->peak_in_use = m.peak;
    stats->reserved = m.reserved;
    return APML_OK;
}

apml_status apml_reset_peak_memory(void)
{
    Memory &m = mem();
    std::lock_guard<std::mutex> lk(m.mu);
    m.peak = m.in_use;
    return APML_OK;
}

apml_status apml_release_cached_memory(void)
{
    Memory &m = mem();
    std::lock_guard<std::mutex> lk(m.mu);
    if (m.free_blocks.empty())
        return APML_OK;
    HIP_TRY(hipDeviceSynchronize());
    for (auto &kv : m.free_blocks)
        for (auto &blk : kv.second) {
            (void)hipFree(blk.second);
            m.reserved -= (int64_t)m.block_size[blk.second];
            m.block_size.erase(blk.second);
        }
    m.free_blocks.clear();
    return APML_OK;
}

apml_status apml_profile_enable(int32_t on)
{
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    p.on = on != 0;
    return APML_OK;
}

apml_status apml_profile_reset(void)
{
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    for (auto &e : p.pending) {
        (void)hipEventSynchronize(e.b);
        p.spare.push_back(e.a);
        p.spare.push_back(e.b);
    }
    p.pending.clear();
    for (int k = 0; k < APML_N_PHASES; ++k) {
        p.total[k] = 0.0;
        p.count[k] = 0;
    }
    return APML_OK;
}

apml_status apml_profile_read(int32_t n, double *total_ms, int64_t *count)
{
    if (n < 0 || n > APML_N_PHASES || (n > 0 && (!total_ms || !count)))
        return fail(APML_ERR_INVALID_ARG, "need 0 <= n <= APML_N_PHASES and output arrays");
    Profiler &p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    for (auto &e : p.pending) {
        HIP_TRY(hipEventSynchronize(e.b));
        float ms = 0.0f;
        HIP_TRY(hipEventElapsedTime(&ms, e.a, e.b));
        p.total[e.phase] += ms;
        p.count[e.phase] += 1;
        p.spare.push_back(e.a);
        p.spare.push_back(e.b);
    }
    p.pending.clear();
    for (int k = 0; k < n; ++k) {
        total_ms[k] = p.total[k];
        count[k] = p.count[k];
    }
    return APML_OK;
}

const char *apml_phase_name(int32_t phase)
{
    if (phase < 0 || phase >= APML_N_PHASES)
        return "";
    return kPhaseNames[phase];
}

const char *apml_status_string(apml_status status)
{
    switch (status) {
    case APML_OK: return "ok";
    case APML_ERR_INVALID_ARG: return "invalid argument";
    case APML_ERR_UNSUPPORTED: return "unsupported";
    case APML_ERR_OUT_OF_MEMORY: return "out of memory";
    case APML_ERR_DEVICE: return "device error";
    case APML_ERR_INTERNAL: return "internal error";
    }
    return "unknown status";
}

const char *apml_last_error(void) { return g_last_error.c_str(); }

int32_t apml_version(void) { return APML_VERSION; }

} // extern "C"
