// C ABI of the scratchpad: context, window ring, plan/forward/backward state
// machine, write-back thread and flush.  Kernels live in k_*.hip.
//
// Streams.  The caller's stream runs forward and backward.  The library has
// four: the ingest stream sorts and deduplicates window batches (and carries
// large write-back copies), the plan stream runs the query and the commit
// sequence, the move stream runs the miss fill (and, with the staged fill,
// the host-to-device copies of gathered rows), and the copy stream carries
// small device-to-host copies of evicted rows.  Host threads gather missing
// rows into pinned staging (staged fill) and scatter evicted rows into the
// host tables ([Collect] / [Exchange] / [Insert] of Sec. IV-B, with the
// CPU-side work done off the critical path).
//
// Ordering (the RAW dependences of Sec. IV-B, for one plan k in flight while
// batch k-1 trains):
//  1  update(k-1) -> forward(k): forward(k) waits for update(k-1)'s event.
//  2/3 update or fill -> victim read: a victim last used by batch k-1 is packed
//     and refilled only after update(k-1); other victims after update(k-2).
//     The plan itself never evicts a slot any window batch uses.
//  4  host write-back -> later fill of the same row: a row evicted by plan p is
//     not in batches p..p+n_p-1 (the hold window), so before the fill of plan k
//     the host joins every write-back job with p + n_p <= k.
#include <hip/hip_runtime.h>
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <functional>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/scratchpipe.h"
#include "sp_internal.h"

using namespace sp;

namespace {

double host_ms()
{
    return std::chrono::duration<double, std::milli>(
               std::chrono::steady_clock::now().time_since_epoch())
        .count();
}

int bits_for(uint64_t v)  // bits needed to represent v (0 -> 0)
{
    int b = 0;
    while (v) ++b, v >>= 1;
    return b;
}

struct Timer {
    static constexpr int N = 8;
    hipEvent_t b[N]{}, e[N]{};
    bool used[N]{};
    int next = 0;
    double ms = 0;
    int64_t count = 0;
    hipError_t init()
    {
        for (int i = 0; i < N; ++i) {
            hipError_t r = hipEventCreate(&b[i]);
            if (r != hipSuccess) return r;
            r = hipEventCreate(&e[i]);
            if (r != hipSuccess) return r;
        }
        return hipSuccess;
    }
    hipError_t harvest(int i)
    {
        if (!used[i]) return hipSuccess;
        hipError_t r = hipEventSynchronize(e[i]);
        if (r != hipSuccess) return r;
        float x = 0;
        r = hipEventElapsedTime(&x, b[i], e[i]);
        if (r != hipSuccess) return r;
        ms += x;
        ++count;
        used[i] = false;
        return hipSuccess;
    }
    hipError_t begin(hipStream_t s)
    {
        hipError_t r = harvest(next);
        return r != hipSuccess ? r : hipEventRecord(b[next], s);
    }
    hipError_t end(hipStream_t s)
    {
        hipError_t r = hipEventRecord(e[next], s);
        used[next] = true;
        next = (next + 1) % N;
        return r;
    }
    // Event pair for a launch that records its own start/stop (kernel time only).
    hipError_t take(hipEvent_t *b0, hipEvent_t *e0)
    {
        hipError_t r = harvest(next);
        *b0 = b[next];
        *e0 = e[next];
        used[next] = true;
        next = (next + 1) % N;
        return r;
    }
    hipError_t flush()
    {
        for (int i = 0; i < N; ++i) {
            hipError_t r = harvest(i);
            if (r != hipSuccess) return r;
        }
        return hipSuccess;
    }
    void destroy()
    {
        for (int i = 0; i < N; ++i) {
            if (b[i]) hipEventDestroy(b[i]);
            if (e[i]) hipEventDestroy(e[i]);
        }
    }
};

struct Job {
    int64_t ticket = 0;
    hipEvent_t ev = nullptr;
    const float *rows = nullptr;
    const int32_t *keys = nullptr;
    int64_t n = 0;
};

struct TicketHost {
    QueryRows qr{};  // the rows of the plan's query (its entering batches, rebuild)
    const uint32_t *uk[MAX_WINDOW] = {};  // the query's probe arrays
    const int32_t *nu[MAX_WINDOW] = {};
    int64_t ent_len[MAX_WINDOW] = {};  // per probe array: IDs (a bound on its unique keys)
    int32_t stamp = 0;    // the query's stamp
    bool keys_direct = false;  // the query wrote the missing keys to pinned host memory
    int64_t nnz = 0, n_unique = 0, n_chunks = 0, n_multi = 0, n_miss = 0;
    int64_t n_own = 0;  // misses of the planned batch itself (n_miss less prefetched rows)
    bool ev_planned = false;  // the plan recorded ev_planned (event-wait mode at plan time)
    int32_t B = 0;
    int ring = 0;
    int nwin = 0;
};

// A wait of the move stream: on an event, or (ev null) until *addr >= val.
struct Wait {
    hipEvent_t ev = nullptr;
    uint64_t *addr = nullptr;
    uint64_t val = 0;
};

// Everything a plan's fill needs on the move stream: what to wait for, then
// the move kernel (stage each victim's old row, write the missing row into
// its slot), then the fill's event and value.  The caller builds it; the
// mapped fill enqueues it at once, the staged fill hands it to the fill
// thread, which first gathers and copies the rows.
struct MoveJob {
    bool gather = false;   // the staged fill's gather and copies, else the move itself
    int64_t k = 0, n = 0;  // plan, rows to place
    int sl = 0, e = 0;     // staging slot, ticket entry
    int32_t u = 0;
    bool timing = false;
    int nwait = 0;
    Wait wait[MAX_WINDOW + 8];
};

thread_local std::string g_create_error;
// allocations sp_create may still make before one is made to fail (testing
// aid: SP_FAIL_ALLOC_AFTER); negative = no limit
thread_local int64_t g_alloc_budget = -1;

// Host threads that split row copies between them: the scatter of evicted
// rows from pinned staging into the host tables (the CPU-side [Insert] of
// Sec. IV-B) and, with the staged fill, the gather of missing rows from the
// host tables into pinned staging ([Collect]).  Rows sit at random places in
// tables far larger than any cache, so the copies are latency-bound and
// spread over several threads.  The calling thread takes part; work is
// handed out in pieces of `grain` items from a shared counter.  One caller at
// a time (each user owns its pool).
class Pool {
  public:
    void start(int helpers)
    {
        for (int i = 0; i < helpers; ++i) threads_.emplace_back([this] { loop(); });
    }
    // fn(b, e) over [0, n) in pieces; returns when every piece has run.
    template <typename F>
    void run(int64_t n, int64_t grain, F &&fn)
    {
        if (n <= 0) return;
        if (threads_.empty() || n <= grain) {
            fn((int64_t)0, n);
            return;
        }
        Work w{[&fn](int64_t b, int64_t e) { fn(b, e); }, n, grain};
        {
            std::lock_guard<std::mutex> lk(m_);
            work_ = &w;
            ++gen_;
        }
        cv_start_.notify_all();
        take(w);
        std::unique_lock<std::mutex> lk(m_);
        work_ = nullptr;  // helpers that have not joined yet stay out
        cv_done_.wait(lk, [&] { return w.busy == 0; });
    }
    void stop()
    {
        {
            std::lock_guard<std::mutex> lk(m_);
            stop_ = true;
        }
        cv_start_.notify_all();
        for (auto &t : threads_) t.join();
        threads_.clear();
    }
    int helpers() const { return (int)threads_.size(); }

  private:
    struct Work {
        std::function<void(int64_t, int64_t)> fn;
        int64_t n, grain;
        std::atomic<int64_t> next{0};
        int busy = 0;  // helpers inside take(), under m_
    };
    static void take(Work &w)
    {
        for (;;) {
            const int64_t b = w.next.fetch_add(w.grain);
            if (b >= w.n) return;
            w.fn(b, std::min(w.n, b + w.grain));
        }
    }
    void loop()
    {
        int64_t seen = 0;
        for (;;) {
            Work *w;
            {
                std::unique_lock<std::mutex> lk(m_);
                cv_start_.wait(lk, [&] { return gen_ != seen || stop_; });
                if (stop_) return;
                seen = gen_;
                w = work_;
                if (!w) continue;
                ++w->busy;
            }
            take(*w);
            std::lock_guard<std::mutex> lk(m_);
            if (--w->busy == 0) cv_done_.notify_all();
        }
    }
    std::vector<std::thread> threads_;
    std::mutex m_;
    std::condition_variable cv_start_, cv_done_;
    Work *work_ = nullptr;
    int64_t gen_ = 0;
    bool stop_ = false;
};

// Copy one row of `bytes` (a multiple of 16, both ends 16-byte aligned) with
// streaming stores: the destination is not read first and does not displace
// the caches, since nothing reads it again soon (the copy engine reads the
// staging; a table row is read again only when it misses much later).
inline void stream_row(float *dst, const float *src, size_t bytes)
{
    const __m128i *s = reinterpret_cast<const __m128i *>(src);
    __m128i *d = reinterpret_cast<__m128i *>(dst);
    for (size_t k = 0; k < bytes / 16; ++k) _mm_stream_si128(d + k, _mm_loadu_si128(s + k));
}

// Copy rows between host tables and a staging buffer: staging row i holds
// table row keys[i] (table key >> row_bits, row key & mask); negative keys,
// and keys outside the tables, are skipped.  to_tables: scatter staging ->
// tables, else gather.  The rows a few keys ahead are prefetched, so several
// random rows are in flight per thread.  Returns the rows copied.
int64_t copy_rows(float *const *tables, const Tables &tb, int dim, float *stage,
                  const int32_t *keys, int64_t b, int64_t e, bool to_tables)
{
    constexpr int AHEAD = 8;
    const uint32_t mask = (1u << tb.row_bits) - 1u;
    const size_t row_bytes = sizeof(float) * (size_t)dim;
    auto row_of = [&](int32_t key) -> float * {
        if (key < 0) return nullptr;
        const int t = key >> tb.row_bits;
        const int64_t r = key & mask;
        if (t >= tb.T || r >= tb.rows[t]) return nullptr;
        return tables[t] + r * dim;
    };
    for (int64_t i = b; i < std::min(e, b + AHEAD); ++i)
        if (float *row = row_of(keys[i]))
            for (size_t o = 0; o < row_bytes; o += 64)
                _mm_prefetch(reinterpret_cast<const char *>(row) + o, _MM_HINT_T0);
    int64_t w = 0;
    for (int64_t i = b; i < e; ++i) {
        if (i + AHEAD < e) {  // the table row (gather) or staging row (scatter) ahead
            const char *pf = to_tables ? reinterpret_cast<const char *>(stage + (i + AHEAD) * dim)
                                       : reinterpret_cast<const char *>(row_of(keys[i + AHEAD]));
            if (pf)
                for (size_t o = 0; o < row_bytes; o += 64) _mm_prefetch(pf + o, _MM_HINT_T0);
        }
        float *row = row_of(keys[i]);
        if (!row) continue;
        if (to_tables) stream_row(row, stage + i * dim, row_bytes);
        else stream_row(stage + i * dim, row, row_bytes);
        ++w;
    }
    _mm_sfence();  // the streamed rows are visible before the caller hands them on
    return w;
}

}  // namespace

constexpr uint32_t SP_FLAGS_ALL =
    SP_FLAG_DEBUG_SYNC | SP_FLAG_TIMING | SP_FLAG_EVENT_WAITS | SP_FLAG_POISON | SP_FLAG_DEFER_SORTS;

// words of sp_ctx::sem, one cache line apart
constexpr int SEM_PLANNED = 0, SEM_FILLED = 8, SEM_WORDS = 16;
// then, per ring entry e (8 words apart), ticket + 1 of the last update of a
// ticket in entry e: monotonic, since entry e is reused by ticket j + nring
// only after update j has run (its query waits for it)
constexpr int SEM_UPD = SEM_WORDS;
static int sem_words(int nring) { return SEM_UPD + 8 * nring; }

// staging slots of evicted rows (fill of plan p, copy of plan p - 1 and the
// host scatter of plan p - 2 can all be in flight)
constexpr int MAX_NSTAGE = 3;
// staged fill: bytes of gathered rows per host-to-device copy, an eighth of
// the plan's rows within these bounds (measured on an MI355X beside a
// device-to-host copy of the same size: 8 MiB copies reach 45 GB/s, 32 MiB
// copies 56 GB/s; a small fill still needs several copies to overlap its
// gather), and per work item of the gather threads (small, so that all of
// them work on the piece whose copy is next)
constexpr int64_t FILL_PIECE_MIN_BYTES = 8ll << 20;
constexpr int64_t FILL_PIECE_BYTES = 32ll << 20;
constexpr int64_t FILL_ITEM_BYTES = 1ll << 20;
// Host ID arrays from this size on are copied into pinned memory by several
// threads (one reaches a fraction of the host's memory bandwidth).
constexpr int64_t IDCOPY_ABOVE_BYTES = 8ll << 20;
constexpr int64_t IDCOPY_GRAIN_BYTES = 2ll << 20;
// write-back copies above this size go on the ingest stream, where they
// overlap the next fill; smaller ones go on the copy stream
constexpr int64_t SMALL_COPY_BYTES = 8ll << 20;
// A write-back copy above this many bytes keeps the ingest stream busy for
// most of a step (5 ms and more on the host link): batches prepared ahead are
// then sorted behind the update instead of behind it.
constexpr int64_t DEFER_BEHIND_COPY_BYTES = 256ll << 20;
// device-to-host copies of write-backs are issued in pieces of this size
constexpr int64_t WB_PIECE_BYTES = 32ll << 20;

struct sp_ctx {
    // configuration
    int T = 0, D = 0, L = 0, device = 0;
    int policy = POLICY_LRU, P = 0;  // replacement policy, past batches held
    uint64_t seed = 0;
    uint32_t flags = 0;
    int32_t max_batch = 0;
    int64_t max_ids = 0, max_table_ids = 0, nchunk_max = 0;
    int key_bits = 0, chunk = 0;
    Tables tb{};
    int64_t slots[MAX_TABLES]{}, total_slots = 0, maxS = 0;
    // per table: slots fresh[t] .. slots[t] - 1 have never held a row
    int64_t fresh[MAX_TABLES]{};
    float *host[MAX_TABLES]{}, *host_dev[MAX_TABLES]{};

    // device state
    float *storage = nullptr;
    int32_t *key_of_slot = nullptr, *last_use = nullptr;
    int32_t *hold_to = nullptr;  // last plan holding each slot (-1: none)
    int32_t *held = nullptr;     // stamp of the last query whose entering batches hold the slot
    int32_t stamp = 0;           // of the last query
    int64_t total_rows = 0;      // rows of all tables
    int64_t *rbase = nullptr;    // [T + 1] first row index of each table (device)
    int32_t *lastq = nullptr, *pend = nullptr;  // per row: see RowIndex
    int32_t *hcnt = nullptr;     // [MAX_TABLES][HOLD_RING] slots per table and hold_to value
    int64_t entered = -1;        // last batch whose slots an accepted plan has marked held
    // the last plan with misses took them all from never-used slots (so it
    // wrote nothing back)
    bool last_fresh = true;
    int32_t *uses = nullptr;  // per-slot use counts, LFU only
    int pf_depth = 0;         // plans also fill the missing rows of this many successors
    uint32_t *pf_own_key = nullptr;  // prefetch mode: the planned batch's own misses,
    int32_t *pf_own_uidx = nullptr;  // as the query compacts them
    int32_t *pf_flag = nullptr;      // [pf_depth][max_ids] successors' unique keys to prefetch
    uint64_t *hash = nullptr;
    uint32_t hash_mask = 0;
    int64_t hash_used = 0;

    // window ring: batch q lives in entry q % nring (ring_batch[r] = q, -1 if none)
    int nring = 0;
    std::vector<BatchDev> ring;
    std::vector<int64_t> ring_batch, ring_nnz, ring_B;
    std::vector<hipEvent_t> ring_ready;     // ingest of the entry's batch finished
    std::vector<char> ring_seen;            // the plan stream has waited for ring_ready
    hipEvent_t ev_consumed = nullptr;       // last ingest has read the caller's arrays

    // tickets
    // tickets: plan k uses entry k % nring, like its batch in the window ring,
    // so ev_upd[r] (backward of the entry's ticket issued) also frees ring[r]
    std::vector<TicketDev> tk;
    std::vector<TicketHost> tkh;
    std::vector<hipEvent_t> ev_planned, ev_filled, ev_upd;
    // stream-ordered counters in device memory for the two waits that are
    // nearly always still pending when they are enqueued (a value wait costs
    // the host a fraction of a wait on an unfinished event): sem[SEM_PLANNED]
    // reaches k + 1 when plan k's commit has run, sem[SEM_FILLED] when its
    // fill has.  The events are recorded as well, for SP_FLAG_EVENT_WAITS.
    uint64_t *sem = nullptr;
    std::vector<hipStream_t> upd_stream;    // stream each ticket's backward ran on
    std::vector<char> upd_val;              // its update wrote its SEM_UPD word
    int64_t planned = 0, forwarded = 0, updated = 0;
    // query of plan spec_ticket over spec_nhold batches, issued early by the
    // plan before it (-1: none)
    int64_t spec_ticket = -1;
    int spec_nhold = 0;
    hipStream_t last_update_stream = nullptr;

    // scratch of the plan stream and of the ingest stream
    uint32_t *tmp_k = nullptr, *tmp_v = nullptr, *hist = nullptr;
    ScanWs ws_plan;
    uint32_t *itmp_k = nullptr, *itmp_v = nullptr, *ihist = nullptr;
    ScanWs ws_ingest;
    int32_t *sel_state = nullptr, *sel_hist = nullptr;
    uint32_t *vk0 = nullptr, *vv0 = nullptr, *vk1 = nullptr;
    float *partial = nullptr;
    float *static_partial = nullptr;  // this device's fixed array (sp_backward_update_static)
    DevCounters *cnt = nullptr;
    int32_t *cnt_part = nullptr;  // [PART_COPIES][2 * MAX_TABLES] probe counter copies, then
                                  // the query's arrival count
    // host-coherent copy of the counters, one 64-bit word per counter: query
    // sequence number << 32 | value; and its device address
    uint64_t *h_cnt = nullptr, *h_cnt_dev = nullptr;
    // ingests in LDS report that they have read the caller's arrays through
    // word h_cnt[COUNTER_WORDS]: blocks count themselves in cons_counter
    uint32_t *cons_counter = nullptr;
    uint32_t cons_issued = 0, cons_seq = 0;
    bool wait_cons_event = false, wait_cons_word = false;  // for the sp_plan call in progress
    // staged fill: batches prepared ahead whose ingest sp_backward_update
    // enqueues behind its update (host ones already in their pinned buffers)
    struct Deferred {
        sp_batch bt;
        int64_t q;
    };
    std::vector<Deferred> deferred;
    uint32_t wait_seq = 0;  // the word the last ingest from the caller's arrays writes
    uint32_t qseq = 0;        // sequence number of the last query issued
    uint32_t spec_seq = 0;    // that of the early query

    // write-back staging (two in flight)
    int64_t stage_rows = 0;
    // staging of evicted rows, plan p in slot p % nstage: n rows, then their n
    // previous keys.  Plan p's copy to the host is issued by plan p + 1 (or by
    // flush), when its fill has nearly always finished: copy_pending = p
    float *stage_dev[MAX_NSTAGE]{}, *stage_host[MAX_NSTAGE]{};
    hipEvent_t ev_d2h[MAX_NSTAGE]{};
    int nstage = 3;  // staging slots in use
    int64_t copy_pending = -1, copy_n = 0;

    // plan stream: query, hold, victims, commit; ingest stream: sorting and
    // deduplicating batches as they become visible; move stream: write-back
    // staging and miss fills; copy stream: the device-to-host copy of evicted
    // rows when it is small.  A process gets few hardware queues (four by
    // default) and streams beyond them share one, in order: the copy stream
    // may land behind the fill.  A large copy therefore goes on the ingest
    // stream, where it overlaps the next fill.
    hipStream_t s_plan = nullptr, s_ingest = nullptr, s_move = nullptr, s_copy = nullptr;

    // write-back thread
    std::thread worker;
    std::mutex mu;
    std::condition_variable cv, cv_done;
    std::deque<Job> jobs;
    int64_t done_upto = -1;
    bool stop = false;
    hipError_t worker_err = hipSuccess;
    std::deque<std::pair<int64_t, int64_t>> deadlines;  // (ticket, first plan that may refill)
    int64_t wb_evictions = 0, wb_bytes = 0;
    Pool scatter;

    // staged fill (SP_FILL_STAGED): a plan's missing keys come to the host
    // (h_mkey, copied behind the victim choice), host threads gather their
    // rows from the tables into pinned staging (h_fill) and copies take them
    // to the device (d_fill) piece by piece as they are gathered; the move
    // kernel then writes them into their slots.  The fill thread does this
    // per plan, in plan order, and enqueues everything of a plan's fill on the
    // move stream, where the calling thread then enqueues nothing.  Staging
    // slot k % nstage, like the write-back's.
    bool staged = false;
    int32_t *h_mkey[MAX_NSTAGE]{};
    uint32_t *h_mkey_dev[MAX_NSTAGE]{};  // their device-visible addresses
    float *h_fill[MAX_NSTAGE]{}, *d_fill[MAX_NSTAGE]{};
    hipEvent_t ev_mkey[MAX_NSTAGE]{}, ev_fill_h2d[MAX_NSTAGE]{};
    bool fill_h2d_used[MAX_NSTAGE]{};
    std::thread filler;
    std::mutex fmu;
    std::condition_variable fcv, fcv_done;
    std::deque<MoveJob> fjobs;
    int64_t fill_enqueued = 0;  // plans whose fill is fully enqueued: tickets below this
    bool fstop = false;
    std::string fill_err;       // first error of the fill thread (then the context is broken)
    Pool gather;
    Pool idcopy;  // copies of large host ID arrays into pinned memory (calling thread)
    double gather_ms = 0, fill_join_ms = 0;
    Timer t_h2d;
    bool poison = false;

    // pinned copies of window arrays handed over in host memory, per ring
    // entry: the caller's arrays are copied here on the host, then to the
    // device asynchronously (ev_ids: that copy has run)
    std::vector<int32_t *> h_ids, h_off;
    std::vector<hipEvent_t> ev_ids;
    std::vector<char> ids_pending;

    // bookkeeping
    sp_stats st{};
    Timer t_fwd, t_bwd, t_cmb, t_plan, t_fill, t_ing, t_qry;
    int64_t dev_bytes = 0, pinned_bytes = 0;
    // sp_plan: ingest, query, wait, commit, mover, waiting for inputs to be read
    double host_ms[6] = {0, 0, 0, 0, 0, 0};
    std::vector<void *> dev_allocs, pinned_allocs;
    std::string err;
    bool broken = false;
};

// ---------------------------------------------------------------- error helpers

static sp_status fail(sp_ctx *h, sp_status code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (h) {
        h->err = buf;
        if (code == SP_ERR_HIP) h->broken = true;
    } else {
        g_create_error = buf;
    }
    return code;
}

#define HIPCHK(h, call)                                                                        \
    do {                                                                                       \
        hipError_t _e = (call);                                                                \
        if (_e != hipSuccess)                                                                  \
            return fail((h), SP_ERR_HIP, "%s failed: %s (%s:%d)", #call, hipGetErrorString(_e), \
                        __FILE__, __LINE__);                                                   \
    } while (0)

#define CHECK_LAUNCH(h) HIPCHK(h, hipGetLastError())

static sp_status usable(sp_ctx *h)
{
    if (!h) return SP_ERR_STATE;
    if (h->broken) return fail(h, SP_ERR_STATE, "context unusable after an earlier HIP error");
    hipError_t e = hipSetDevice(h->device);
    if (e != hipSuccess) return fail(h, SP_ERR_HIP, "hipSetDevice: %s", hipGetErrorString(e));
    return SP_OK;
}

// True when the allocation budget of SP_FAIL_ALLOC_AFTER is spent.
static bool injected_alloc_failure()
{
    if (g_alloc_budget == 0) return true;
    if (g_alloc_budget > 0) --g_alloc_budget;
    return false;
}

template <typename T>
static sp_status dalloc(sp_ctx *h, T **p, int64_t count)
{
    size_t bytes = (size_t)std::max<int64_t>(count, 1) * sizeof(T);
    if (injected_alloc_failure()) {
        *p = nullptr;
        return fail(h, SP_ERR_OOM, "hipMalloc(%zu) failed: injected (SP_FAIL_ALLOC_AFTER)", bytes);
    }
    hipError_t e = hipMalloc((void **)p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return fail(h, SP_ERR_OOM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    }
    h->dev_allocs.push_back((void *)*p);
    h->dev_bytes += (int64_t)bytes;
    return SP_OK;
}

template <typename T>
static sp_status palloc(sp_ctx *h, T **p, int64_t count)
{
    size_t bytes = (size_t)std::max<int64_t>(count, 1) * sizeof(T);
    if (injected_alloc_failure()) {
        *p = nullptr;
        return fail(h, SP_ERR_OOM, "hipHostMalloc(%zu) failed: injected (SP_FAIL_ALLOC_AFTER)", bytes);
    }
    hipError_t e = hipHostMalloc((void **)p, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return fail(h, SP_ERR_OOM, "hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    }
    h->pinned_allocs.push_back((void *)*p);
    h->pinned_bytes += (int64_t)bytes;
    return SP_OK;
}

#define TRY(x)                          \
    do {                                \
        sp_status _s = (x);             \
        if (_s != SP_OK) return _s;     \
    } while (0)

// ---------------------------------------------------------------- write-back thread

static void worker_main(sp_ctx *h)
{
    (void)hipSetDevice(h->device);
    const size_t row_bytes = sizeof(float) * (size_t)h->D;
    for (;;) {
        Job j;
        {
            std::unique_lock<std::mutex> lk(h->mu);
            h->cv.wait(lk, [&] { return !h->jobs.empty() || h->stop; });
            if (h->jobs.empty()) return;
            j = h->jobs.front();
        }
        int64_t ev = 0;
        if (j.n > 0) {
            hipError_t e = hipEventSynchronize(j.ev);
            if (e != hipSuccess) {
                std::lock_guard<std::mutex> lk(h->mu);
                h->worker_err = e;
            } else {
                std::atomic<int64_t> wr{0};
                h->scatter.run(j.n, 512, [&](int64_t b, int64_t e2) {
                    wr += copy_rows(h->host, h->tb, h->D, const_cast<float *>(j.rows), j.keys,
                                    b, e2, true);
                });
                ev = wr.load();
            }
        }
        {
            std::lock_guard<std::mutex> lk(h->mu);
            h->jobs.pop_front();
            h->done_upto = j.ticket;
            h->wb_evictions += ev;
            h->wb_bytes += ev * (int64_t)row_bytes;
        }
        h->cv_done.notify_all();
    }
}

static sp_status join_jobs(sp_ctx *h, int64_t upto)
{
    std::unique_lock<std::mutex> lk(h->mu);
    h->cv_done.wait(lk, [&] { return h->done_upto >= upto || h->worker_err != hipSuccess; });
    if (h->worker_err != hipSuccess)
        return fail(h, SP_ERR_HIP, "write-back thread: %s", hipGetErrorString(h->worker_err));
    return SP_OK;
}

// ---------------------------------------------------------------- fixed scratch

// Device address of the fixed partial-sum array on each device, taken once
// per device with that device current (each device has its own copy).
static std::mutex g_static_mu;
static void *g_static_partial[256];

static sp_status static_partial_for(sp_ctx *h, int device, float **out)
{
    if (device < 0 || device >= 256) return fail(h, SP_ERR_INVALID_ARG, "device %d out of range", device);
    std::lock_guard<std::mutex> lk(g_static_mu);
    if (!g_static_partial[device]) {
        void *p = nullptr;
        const hipError_t e = static_partial_address(&p);
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(h, SP_ERR_HIP, "hipGetSymbolAddress(fixed partial array): %s",
                        hipGetErrorString(e));
        }
        g_static_partial[device] = p;
    }
    *out = (float *)g_static_partial[device];
    return SP_OK;
}

// ---------------------------------------------------------------- fill

// Enqueue a plan's fill on the move stream: its waits, the move kernel
// (rows from the mapped host tables, or from `staged` device rows), then the
// fill's event and counter value.  Called by the calling thread (mapped fill)
// or the fill thread (staged fill), never by both for one context.
static hipError_t enqueue_move(sp_ctx *h, const MoveJob &j, const float *staged)
{
    hipStream_t s = h->s_move;
    hipError_t r = hipSuccess;
    for (int i = 0; i < j.nwait && r == hipSuccess; ++i) {
        const Wait &w = j.wait[i];
        r = w.ev ? hipStreamWaitEvent(s, w.ev, 0)
                 : hipStreamWaitValue64(s, w.addr, w.val, hipStreamWaitValueGte, ~0ull);
    }
    if (r != hipSuccess) return r;
    if (j.n > 0) {
        if (j.timing && (r = h->t_fill.begin(s)) != hipSuccess) return r;  // the kernel itself
        launch_move(h->storage, h->D, h->tb, h->host_dev, h->tk[j.e], j.n, j.u, h->stage_dev[j.sl],
                    staged, s);
        if ((r = hipGetLastError()) != hipSuccess) return r;
        if (j.timing && (r = h->t_fill.end(s)) != hipSuccess) return r;
        if (staged && h->poison)  // the staging is spent: any later read of it shows
            launch_fill_i32((int32_t *)h->d_fill[j.sl], j.n * h->D, 0x7FC00000, s);
    }
    if ((r = hipEventRecord(h->ev_filled[j.e], s)) != hipSuccess) return r;
    return hipStreamWriteValue64(s, h->sem + SEM_FILLED, (uint64_t)j.k + 1, 0);
}

// The staged fill's gather of one plan, on the fill thread: wait for the
// missing keys on the host, then the gather threads take small items of them
// in turn and gather their rows into pinned staging; the thread that
// completes the last item of a piece enqueues that piece's copy to the device
// (pieces are independent, so their copies may be enqueued in any order; the
// move is enqueued after all of them).
static hipError_t staged_gather(sp_ctx *h, const MoveJob &j)
{
    const int sl = j.sl;
    hipError_t r = hipSuccess;
    if (j.n <= 0) return r;
    if ((r = hipEventSynchronize(h->ev_mkey[sl])) != hipSuccess) return r;
    // the copies out of this pinned staging slot (plan k - nstage) have run
    if (h->fill_h2d_used[sl] && (r = hipEventSynchronize(h->ev_fill_h2d[sl])) != hipSuccess)
        return r;
    const double t0 = host_ms();
    const int D = h->D;
    const int64_t item = std::max<int64_t>(1, FILL_ITEM_BYTES / (4 * (int64_t)D));
    const int64_t piece_bytes =
        std::clamp<int64_t>(j.n * 4 * (int64_t)D / 8, FILL_PIECE_MIN_BYTES, FILL_PIECE_BYTES);
    const int64_t piece = std::max<int64_t>(1, piece_bytes / (4 * (int64_t)D) / item) * item;
    const int64_t nitems = (j.n + item - 1) / item, npieces = (j.n + piece - 1) / piece;
    std::unique_ptr<std::atomic<int64_t>[]> left(new std::atomic<int64_t>[npieces]);
    for (int64_t q = 0; q < npieces; ++q)  // items of piece q
        left[q] = (std::min(j.n, (q + 1) * piece) - q * piece + item - 1) / item;
    float *const hs = h->h_fill[sl];
    if (j.timing && (r = h->t_h2d.begin(h->s_move)) != hipSuccess) return r;
    std::atomic<int> bad{0};
    h->gather.run(nitems, 1, [&](int64_t i0, int64_t i1) {
        for (int64_t i = i0; i < i1; ++i) {
            const int64_t b = i * item, e = std::min(j.n, b + item);
            copy_rows(h->host, h->tb, D, hs, h->h_mkey[sl], b, e, false);
            const int64_t q = b / piece;
            if (left[q].fetch_sub(1) != 1) continue;
            // the piece is complete (copy_rows fenced its streamed stores)
            (void)hipSetDevice(h->device);
            const int64_t pb = q * piece, pe = std::min(j.n, pb + piece);
            const hipError_t c = hipMemcpyAsync(h->d_fill[sl] + pb * D, hs + pb * D,
                                                sizeof(float) * (pe - pb) * D,
                                                hipMemcpyHostToDevice, h->s_move);
            if (c != hipSuccess) bad.store((int)c);
        }
    });
    if (bad.load()) return (hipError_t)bad.load();
    if (j.timing && (r = h->t_h2d.end(h->s_move)) != hipSuccess) return r;
    if ((r = hipEventRecord(h->ev_fill_h2d[sl], h->s_move)) != hipSuccess) return r;
    h->fill_h2d_used[sl] = true;
    h->gather_ms += host_ms() - t0;
    return r;
}

static void filler_main(sp_ctx *h)
{
    (void)hipSetDevice(h->device);
    for (;;) {
        MoveJob j;
        {
            std::unique_lock<std::mutex> lk(h->fmu);
            h->fcv.wait(lk, [&] { return !h->fjobs.empty() || h->fstop; });
            if (h->fjobs.empty()) return;
            j = h->fjobs.front();
        }
        hipError_t r = hipSuccess;
        bool failed;
        {
            std::lock_guard<std::mutex> lk(h->fmu);
            failed = !h->fill_err.empty();
        }
        if (!failed) r = j.gather ? staged_gather(h, j) : enqueue_move(h, j, h->d_fill[j.sl]);
        {
            std::lock_guard<std::mutex> lk(h->fmu);
            if (r != hipSuccess && h->fill_err.empty())
                h->fill_err = std::string("fill of plan ") + std::to_string(j.k) + ": " +
                              hipGetErrorString(r);
            h->fjobs.pop_front();
            if (!j.gather) h->fill_enqueued = j.k + 1;
        }
        h->fcv_done.notify_all();
    }
}

// Wait until the fill thread has enqueued the fill of plan k (staged fill;
// nothing to wait for otherwise).
static sp_status join_fill(sp_ctx *h, int64_t k)
{
    if (!h->staged || k < 0) return SP_OK;
    const double t0 = host_ms();
    std::unique_lock<std::mutex> lk(h->fmu);
    h->fcv_done.wait(lk, [&] { return h->fill_enqueued > k || !h->fill_err.empty(); });
    h->fill_join_ms += host_ms() - t0;
    if (!h->fill_err.empty()) {
        const std::string m = h->fill_err;
        lk.unlock();
        return fail(h, SP_ERR_HIP, "%s", m.c_str());
    }
    return SP_OK;
}

// ---------------------------------------------------------------- create / destroy

static void release(sp_ctx *h)
{
    if (!h) return;
    if (h->filler.joinable()) {  // it enqueues what is queued, then ends
        {
            std::lock_guard<std::mutex> lk(h->fmu);
            h->fstop = true;
        }
        h->fcv.notify_all();
        h->filler.join();
    }
    h->gather.stop();
    if (h->worker.joinable()) {
        {
            std::lock_guard<std::mutex> lk(h->mu);
            h->stop = true;
        }
        h->cv.notify_all();
        h->worker.join();
    }
    h->scatter.stop();
    h->idcopy.stop();
    (void)hipDeviceSynchronize();
    for (auto *v : {&h->ring_ready, &h->ev_planned, &h->ev_filled, &h->ev_upd})
        for (auto &e : *v)
            if (e) hipEventDestroy(e);
    if (h->ev_consumed) hipEventDestroy(h->ev_consumed);
    for (int i = 0; i < MAX_NSTAGE; ++i)
        for (hipEvent_t e : {h->ev_d2h[i], h->ev_mkey[i], h->ev_fill_h2d[i]})
            if (e) hipEventDestroy(e);
    for (hipEvent_t e : h->ev_ids)
        if (e) hipEventDestroy(e);
    h->t_h2d.destroy();
    h->t_fwd.destroy();
    h->t_bwd.destroy();
    h->t_cmb.destroy();
    h->t_plan.destroy();
    h->t_fill.destroy();
    h->t_ing.destroy();
    h->t_qry.destroy();
    if (h->s_plan) hipStreamDestroy(h->s_plan);
    if (h->s_ingest) hipStreamDestroy(h->s_ingest);
    if (h->s_move) hipStreamDestroy(h->s_move);
    if (h->s_copy) hipStreamDestroy(h->s_copy);
    for (void *p : h->dev_allocs) hipFree(p);
    for (void *p : h->pinned_allocs) hipHostFree(p);
    delete h;
}

static sp_status build(sp_ctx *h, const sp_config *c)
{
    const int T = c->num_tables;
    h->T = T;
    h->D = c->dim;
    h->L = c->lookahead;
    h->policy = c->policy;
    h->P = c->hold_past;
    h->pf_depth = std::min(c->prefetch, c->lookahead);  // only window batches are fetched
    h->seed = c->seed;
    h->device = c->device;
    h->flags = c->flags;
    h->max_batch = c->max_batch;
    h->max_ids = c->max_ids;
    h->max_table_ids = c->max_table_ids;
    h->chunk = chunk_positions(h->D);
    int64_t max_rows = 1;
    h->tb.T = T;
    h->tb.slot_base[0] = 0;
    for (int t = 0; t < T; ++t) {
        h->tb.rows[t] = c->rows[t];
        h->slots[t] = c->slots[t];
        h->tb.slot_base[t + 1] = h->tb.slot_base[t] + c->slots[t];
        max_rows = std::max<int64_t>(max_rows, c->rows[t]);
        h->maxS = std::max<int64_t>(h->maxS, c->slots[t]);
    }
    h->total_slots = h->tb.slot_base[T];
    h->tb.row_bits = std::max(1, bits_for((uint64_t)(max_rows - 1)));
    h->key_bits = bits_for((uint64_t)(T - 1)) + h->tb.row_bits;
    if (h->key_bits > 31) return fail(nullptr, SP_ERR_INVALID_ARG, "tables x rows need %d key bits (max 31)", h->key_bits);

    h->staged = c->fill == SP_FILL_STAGED;
    h->poison = (c->flags & SP_FLAG_POISON) != 0;
    HIPCHK(nullptr, hipSetDevice(h->device));
    TRY(static_partial_for(h, h->device, &h->static_partial));
    for (int t = 0; t < T; ++t) {
        h->host[t] = c->host_tables[t];
        if (h->staged) continue;  // read on the host only
        hipPointerAttribute_t attr;
        hipError_t e = hipPointerGetAttributes(&attr, (const void *)c->host_tables[t]);
        void *dp = nullptr;
        if (e == hipSuccess) e = hipHostGetDevicePointer(&dp, (void *)c->host_tables[t], 0);
        if (e != hipSuccess || !dp) {
            (void)hipGetLastError();
            return fail(nullptr, SP_ERR_INVALID_ARG,
                        "host table %d is not pinned, device-mapped memory (use sp_host_alloc)", t);
        }
        h->host_dev[t] = (float *)dp;
    }

    const int64_t S = h->total_slots, N = h->max_ids, TB1 = (int64_t)T * h->max_batch + 1;
    // misses of one plan: the planned batch's, plus its successors' when prefetching
    const int64_t NM = (1 + (int64_t)h->pf_depth) * N;
    const int64_t nchunk_max = N + N / h->chunk + 1;
    h->nchunk_max = nchunk_max;
    TRY(dalloc(h, &h->storage, S * h->D));
    TRY(dalloc(h, &h->key_of_slot, S));
    TRY(dalloc(h, &h->last_use, S));
    TRY(dalloc(h, &h->hold_to, S));
    TRY(dalloc(h, &h->held, S));
    for (int t = 0; t < T; ++t) h->total_rows += h->tb.rows[t];
    TRY(dalloc(h, &h->rbase, T + 1));
    TRY(dalloc(h, &h->lastq, h->total_rows));
    TRY(dalloc(h, &h->pend, h->total_rows));
    TRY(dalloc(h, &h->hcnt, (int64_t)MAX_TABLES * HOLD_RING));
    if (h->policy == POLICY_LFU) TRY(dalloc(h, &h->uses, S));
    int64_t cap = 1024;
    while (cap < 2 * S) cap <<= 1;
    if (cap > (int64_t)1 << 32) return fail(nullptr, SP_ERR_INVALID_ARG, "too many slots");
    h->hash_mask = (uint32_t)(cap - 1);
    TRY(dalloc(h, &h->hash, cap));

    // batches k-max(1, P) (training, or held as past) .. k+L+SP_MAX_AHEAD
    // (prepared) plus one of slack
    h->nring = h->L + 3 + SP_MAX_AHEAD + std::max(0, h->P - 1);
    h->ring.resize(h->nring);
    h->ring_batch.assign(h->nring, -1);
    h->ring_nnz.assign(h->nring, 0);
    h->ring_B.assign(h->nring, 0);
    h->ring_ready.assign(h->nring, nullptr);
    h->ring_seen.assign(h->nring, 0);
    h->tk.assign(h->nring, TicketDev{});
    h->tkh.assign(h->nring, TicketHost{});
    h->ev_planned.assign(h->nring, nullptr);
    h->ev_filled.assign(h->nring, nullptr);
    h->ev_upd.assign(h->nring, nullptr);
    h->upd_stream.assign(h->nring, nullptr);
    h->upd_val.assign(h->nring, 0);
    for (int r = 0; r < h->nring; ++r) {
        BatchDev &b = h->ring[r];
        TRY(dalloc(h, &b.ids, N));
        TRY(dalloc(h, &b.bag_off, TB1));
        TRY(dalloc(h, &b.bag_of, N));
        TRY(dalloc(h, &b.skeys, N));
        TRY(dalloc(h, &b.perm, N));
        TRY(dalloc(h, &b.sbag, N));
        TRY(dalloc(h, &b.ukeys, N));
        TRY(dalloc(h, &b.eslot, N));
        TRY(dalloc(h, &b.inv, N));
        TRY(dalloc(h, &b.seg_off, N + 1));
        TRY(dalloc(h, &b.seg_chunk0, N));
        TRY(dalloc(h, &b.chunk_desc, nchunk_max));
        TRY(dalloc(h, &b.multi, multi_capacity(N, h->chunk)));
        TRY(dalloc(h, &b.scal, T + 3));
        HIPCHK(nullptr, hipEventCreateWithFlags(&h->ring_ready[r], hipEventDisableTiming));
    }
    h->h_ids.assign(h->nring, nullptr);
    h->h_off.assign(h->nring, nullptr);
    h->ev_ids.assign(h->nring, nullptr);
    h->ids_pending.assign(h->nring, 0);
    for (int r = 0; r < h->nring; ++r) {
        TRY(palloc(h, &h->h_ids[r], N));
        TRY(palloc(h, &h->h_off[r], TB1));
        HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_ids[r], hipEventDisableTiming));
    }
    for (int k = 0; k < h->nring; ++k) {
        TicketDev &t = h->tk[k];
        TRY(dalloc(h, &t.hit, N));
        TRY(dalloc(h, &t.slot_u, N));
        TRY(dalloc(h, &t.slot_of, N));
        TRY(dalloc(h, &t.m_key, NM));
        TRY(dalloc(h, &t.m_uidx, NM));
        TRY(dalloc(h, &t.v_slot, NM));
        TRY(dalloc(h, &t.v_old_key, NM));
        TRY(dalloc(h, &t.v_old_lu, NM));
        HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_planned[k], hipEventDisableTiming));
        HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_filled[k], hipEventDisableTiming));
        HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_upd[k], hipEventDisableTiming));
    }
    TRY(dalloc(h, &h->tmp_k, N));
    TRY(dalloc(h, &h->tmp_v, N));
    TRY(dalloc(h, &h->itmp_k, N));
    TRY(dalloc(h, &h->itmp_v, N));
    TRY(dalloc(h, &h->vk0, NM));
    TRY(dalloc(h, &h->vv0, NM));
    TRY(dalloc(h, &h->vk1, NM));
    TRY(dalloc(h, &h->hist, radix_hist_entries(NM)));
    if (h->pf_depth > 0) {
        TRY(dalloc(h, &h->pf_own_key, N));
        TRY(dalloc(h, &h->pf_own_uidx, N));
        TRY(dalloc(h, &h->pf_flag, (int64_t)h->pf_depth * N));
    }
    TRY(dalloc(h, &h->ihist, radix_hist_entries(N)));
    TRY(dalloc(h, &h->cnt, 1));
    TRY(dalloc(h, &h->cnt_part, (int64_t)PART_COPIES * PART_WORDS + 1));
    {
        // scans: victims (tables x slots per table), misses and batches (N),
        // radix histogram tables (at most N + 2048 entries)
        // (and the query's tiles of unique keys, and the LDS ingest's workgroups)
        const int64_t tiles = std::max({scan_tiles(T, h->maxS), scan_tiles(1, NM + 4096),
                                        (N + QUERY_TILE - 1) / QUERY_TILE,
                                        (int64_t)T * ingest_splits(T)}) + 2;
        for (ScanWs *ws : {&h->ws_plan, &h->ws_ingest}) {
            ws->max_tiles = tiles;
            TRY(dalloc(h, &ws->status, LB_WORDS * tiles));
            TRY(dalloc(h, &ws->counter, 1));
            ws->err = &h->cnt->err_sticky;
        }
    }
    TRY(dalloc(h, &h->sel_state, 3 * MAX_TABLES));  // v* prefix, slots to take, arrivals
    TRY(dalloc(h, &h->sel_hist, (int64_t)MAX_TABLES * SEL_BINS));
    TRY(dalloc(h, &h->partial, nchunk_max * h->D));
    h->stage_rows = std::min<int64_t>(NM, S);
    h->nstage = MAX_NSTAGE;
    for (int i = 0; i < h->nstage; ++i) {
        TRY(dalloc(h, &h->stage_dev[i], h->stage_rows * (h->D + 1)));
        TRY(palloc(h, &h->stage_host[i], h->stage_rows * (h->D + 1)));
        HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_d2h[i], hipEventDisableTiming));
        if (h->staged) {  // at most min(misses, slots) rows per plan, like the write-back
            {  // device-mapped: the query writes the missing keys here itself
                void *p = nullptr;
                const size_t bytes = sizeof(int32_t) * (size_t)std::max<int64_t>(h->stage_rows, 1);
                if (injected_alloc_failure())
                    return fail(h, SP_ERR_OOM, "hipHostMalloc(%zu) failed: injected (SP_FAIL_ALLOC_AFTER)", bytes);
                hipError_t e = hipHostMalloc(&p, bytes, hipHostMallocMapped);
                if (e != hipSuccess) {
                    (void)hipGetLastError();
                    return fail(h, SP_ERR_OOM, "hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
                }
                h->pinned_allocs.push_back(p);
                h->pinned_bytes += (int64_t)bytes;
                h->h_mkey[i] = (int32_t *)p;
                HIPCHK(nullptr, hipHostGetDevicePointer((void **)&h->h_mkey_dev[i], p, 0));
            }
            TRY(palloc(h, &h->h_fill[i], h->stage_rows * h->D));
            TRY(dalloc(h, &h->d_fill[i], h->stage_rows * h->D));
            HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_mkey[i], hipEventDisableTiming));
            HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_fill_h2d[i], hipEventDisableTiming));
        }
    }
    {
        void *p = nullptr;
        const size_t bytes = sizeof(uint64_t) * (COUNTER_WORDS + 1);
        if (injected_alloc_failure())
            return fail(h, SP_ERR_OOM, "hipHostMalloc(counters) failed: injected (SP_FAIL_ALLOC_AFTER)");
        hipError_t e = hipHostMalloc(&p, bytes, hipHostMallocMapped | hipHostMallocCoherent);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(h, SP_ERR_OOM, "hipHostMalloc(counters): %s", hipGetErrorString(e));
        }
        h->pinned_allocs.push_back(p);
        h->h_cnt = (uint64_t *)p;
        memset(p, 0, bytes);
        HIPCHK(nullptr, hipHostGetDevicePointer((void **)&h->h_cnt_dev, p, 0));
    }

    TRY(dalloc(h, &h->cons_counter, 1));
    TRY(dalloc(h, &h->sem, sem_words(h->nring)));
    HIPCHK(nullptr, hipEventCreateWithFlags(&h->ev_consumed, hipEventDisableTiming));
    HIPCHK(nullptr, hipStreamCreateWithFlags(&h->s_plan, hipStreamNonBlocking));
    HIPCHK(nullptr, hipStreamCreateWithFlags(&h->s_ingest, hipStreamNonBlocking));
    HIPCHK(nullptr, hipStreamCreateWithFlags(&h->s_move, hipStreamNonBlocking));
    HIPCHK(nullptr, hipStreamCreateWithFlags(&h->s_copy, hipStreamNonBlocking));
    HIPCHK(nullptr, h->t_fwd.init());
    HIPCHK(nullptr, h->t_bwd.init());
    HIPCHK(nullptr, h->t_cmb.init());
    HIPCHK(nullptr, h->t_plan.init());
    HIPCHK(nullptr, h->t_fill.init());
    HIPCHK(nullptr, h->t_ing.init());
    HIPCHK(nullptr, h->t_qry.init());
    HIPCHK(nullptr, h->t_h2d.init());

    // initial state: nothing cached
    HIPCHK(nullptr, hipMemsetAsync(h->cons_counter, 0, sizeof(uint32_t), h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->sem, 0, sizeof(uint64_t) * sem_words(h->nring), h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->key_of_slot, 0xFF, sizeof(int32_t) * S, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->last_use, 0xFF, sizeof(int32_t) * S, h->s_plan));
    if (h->uses) HIPCHK(nullptr, hipMemsetAsync(h->uses, 0, sizeof(int32_t) * S, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->hold_to, 0xFF, sizeof(int32_t) * S, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->held, 0, sizeof(int32_t) * S, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->lastq, 0xFF, sizeof(int32_t) * h->total_rows, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->pend, 0, sizeof(int32_t) * h->total_rows, h->s_plan));
    {
        std::vector<int64_t> rb((size_t)T + 1, 0);
        for (int t = 0; t < T; ++t) rb[t + 1] = rb[t] + h->tb.rows[t];
        HIPCHK(nullptr, hipMemcpy(h->rbase, rb.data(), sizeof(int64_t) * (T + 1), hipMemcpyHostToDevice));
    }
    HIPCHK(nullptr, hipMemsetAsync(h->hcnt, 0, sizeof(int32_t) * MAX_TABLES * HOLD_RING, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->hash, 0xFF, sizeof(uint64_t) * cap, h->s_plan));
    // all-ones words are NaN: under SP_FLAG_POISON a read of a never-filled slot shows
    HIPCHK(nullptr, hipMemsetAsync(h->storage, h->poison ? 0xFF : 0, sizeof(float) * S * h->D, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->sel_hist, 0, sizeof(int32_t) * MAX_TABLES * SEL_BINS, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->sel_state, 0, sizeof(int32_t) * 3 * MAX_TABLES, h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->cnt, 0, sizeof(DevCounters), h->s_plan));
    HIPCHK(nullptr, hipMemsetAsync(h->cnt_part, 0, sizeof(int32_t) * (PART_COPIES * PART_WORDS + 1), h->s_plan));
    for (ScanWs *ws : {&h->ws_plan, &h->ws_ingest}) {
        HIPCHK(nullptr, hipMemsetAsync(ws->status, 0, sizeof(uint64_t) * LB_WORDS * ws->max_tiles, h->s_plan));
        HIPCHK(nullptr, hipMemsetAsync(ws->counter, 0, sizeof(uint32_t), h->s_plan));
    }
    HIPCHK(nullptr, hipStreamSynchronize(h->s_plan));
    h->st.min_capacity_margin = INT64_MAX;
    // host copy threads, their calling threads included: the write-back
    // scatter takes half of the cores; with the staged fill the gather, which
    // is on the step's path, takes three quarters and the scatter, which has
    // a few steps to finish, one quarter
    const int hw = (int)std::max(4u, std::thread::hardware_concurrency());
    h->scatter.start(std::max(1, (h->staged ? hw / 4 : std::min(8, hw / 2)) - 1));
    h->worker = std::thread(worker_main, h);
    if (h->staged) {
        h->gather.start(std::max(1, hw * 12 / 16 - 1));
        h->filler = std::thread(filler_main, h);
    }
    // batches of host IDs larger than a single thread copies quickly
    if (h->max_ids * (int64_t)sizeof(int32_t) >= IDCOPY_ABOVE_BYTES)
        h->idcopy.start(std::min(3, std::max(1, hw / 4)));
    return SP_OK;
}

extern "C" sp_status sp_create(const sp_config *c, sp_handle *out)
{
    if (!c || !out) return fail(nullptr, SP_ERR_INVALID_ARG, "null config or output");
    const int T = c->num_tables;
    if (T < 1 || T > MAX_TABLES) return fail(nullptr, SP_ERR_INVALID_ARG, "num_tables %d not in 1..%d", T, MAX_TABLES);
    if (!c->rows || !c->slots || !c->host_tables) return fail(nullptr, SP_ERR_INVALID_ARG, "null rows/slots/host_tables");
    const int D = c->dim;
    if (D < 4 || D > 256 || (D & (D - 1)) != 0)
        return fail(nullptr, SP_ERR_INVALID_ARG, "dim %d must be a power of two in 4..256", D);
    if (c->lookahead < 0 || c->lookahead >= MAX_WINDOW)
        return fail(nullptr, SP_ERR_INVALID_ARG, "lookahead %d not in 0..%d", c->lookahead, MAX_WINDOW - 1);
    if (c->policy < POLICY_LRU || c->policy > POLICY_RANDOM)
        return fail(nullptr, SP_ERR_INVALID_ARG, "unknown policy %d", c->policy);
    if (c->hold_past < 0 || c->hold_past > SP_MAX_HOLD_PAST || c->lookahead + 1 + c->hold_past > MAX_WINDOW)
        return fail(nullptr, SP_ERR_INVALID_ARG, "hold_past %d not in 0..%d with lookahead + 1 + hold_past <= %d",
                    c->hold_past, SP_MAX_HOLD_PAST, MAX_WINDOW);
    if (c->max_table_ids < 0) return fail(nullptr, SP_ERR_INVALID_ARG, "max_table_ids %lld < 0", (long long)c->max_table_ids);
    static_assert(SP_MAX_PREFETCH == MAX_PF, "prefetch bound");
    if (c->prefetch < 0 || c->prefetch > SP_MAX_PREFETCH)
        return fail(nullptr, SP_ERR_INVALID_ARG, "prefetch %d not in 0..%d", c->prefetch,
                    SP_MAX_PREFETCH);
    if (c->fill != SP_FILL_MAPPED && c->fill != SP_FILL_STAGED)
        return fail(nullptr, SP_ERR_INVALID_ARG, "fill %d not SP_FILL_MAPPED or SP_FILL_STAGED", c->fill);
    if (c->max_batch < 0 || c->max_ids < 0 || c->max_ids > INT32_MAX - 1)
        return fail(nullptr, SP_ERR_INVALID_ARG, "bad max_batch / max_ids");
    if ((int64_t)T * c->max_batch + 1 > INT32_MAX) return fail(nullptr, SP_ERR_INVALID_ARG, "too many bags");
    // the backward addresses the [T*B][D] gradients with 32-bit byte offsets
    if ((int64_t)T * c->max_batch * D * 4 > (int64_t)UINT32_MAX)
        return fail(nullptr, SP_ERR_INVALID_ARG, "num_tables * max_batch * dim * 4 bytes exceeds 4 GiB");
    int64_t total = 0;
    for (int t = 0; t < T; ++t) {
        if (c->rows[t] < 1 || c->rows[t] > ((int64_t)1 << 25))
            return fail(nullptr, SP_ERR_INVALID_ARG, "rows[%d]=%lld not in 1..2^25", t, (long long)c->rows[t]);
        if (c->slots[t] < 1 || c->slots[t] > c->rows[t])
            return fail(nullptr, SP_ERR_INVALID_ARG, "slots[%d]=%lld not in 1..rows", t, (long long)c->slots[t]);
        if (!c->host_tables[t]) return fail(nullptr, SP_ERR_INVALID_ARG, "host_tables[%d] is null", t);
        if ((uintptr_t)c->host_tables[t] % 16)
            return fail(nullptr, SP_ERR_INVALID_ARG, "host_tables[%d] is not 16-byte aligned", t);
        total += c->slots[t];
    }
    if (total > INT32_MAX) return fail(nullptr, SP_ERR_INVALID_ARG, "total slots exceed 2^31-1");
    if (c->flags & ~SP_FLAGS_ALL) return fail(nullptr, SP_ERR_INVALID_ARG, "unknown flags");
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || c->device < 0 || c->device >= ndev) {
        (void)hipGetLastError();
        return fail(nullptr, SP_ERR_INVALID_ARG, "device %d not available (%d devices)", c->device, ndev);
    }
    {  // testing aid: fail the allocation after the first n
        const char *f = getenv("SP_FAIL_ALLOC_AFTER");
        g_alloc_budget = f && *f ? std::max<int64_t>(0, strtoll(f, nullptr, 10)) : -1;
    }
    sp_ctx *h = new sp_ctx();
    sp_status s = build(h, c);
    g_alloc_budget = -1;
    if (s != SP_OK) {
        if (!h->err.empty()) g_create_error = h->err;
        release(h);
        return s;
    }
    *out = h;
    return SP_OK;
}

extern "C" void sp_destroy(sp_handle h)
{
    if (!h) return;
    (void)hipSetDevice(h->device);
    release(h);
}

extern "C" const char *sp_last_error(sp_handle h)
{
    return h ? h->err.c_str() : g_create_error.c_str();
}

extern "C" sp_status sp_host_alloc(size_t bytes, void **ptr)
{
    if (!ptr || bytes == 0) return fail(nullptr, SP_ERR_INVALID_ARG, "bad sp_host_alloc arguments");
    hipError_t e = hipHostMalloc(ptr, bytes, hipHostMallocMapped | hipHostMallocPortable);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *ptr = nullptr;
        return fail(nullptr, SP_ERR_OOM, "hipHostMalloc(%zu): %s", bytes, hipGetErrorString(e));
    }
    return SP_OK;
}

extern "C" void sp_host_free(void *ptr)
{
    if (ptr) (void)hipHostFree(ptr);
}

// ---------------------------------------------------------------- plan

// Make stream s wait for event e unless e has already completed: a wait on a
// pending event recorded on another stream costs the host several times more
// than asking whether it has completed.
static hipError_t wait_unless_done(hipStream_t s, hipEvent_t e)
{
    const hipError_t q = hipEventQuery(e);
    if (q == hipSuccess) return hipSuccess;
    if (q != hipErrorNotReady) return q;
    return hipStreamWaitEvent(s, e, 0);
}

// A caller's host array into pinned memory, large ones over the ID copy
// threads.
static void copy_host(sp_ctx *h, void *dst, const void *src, int64_t bytes)
{
    if (bytes < 2 * IDCOPY_GRAIN_BYTES || h->idcopy.helpers() == 0) {
        if (bytes > 0) memcpy(dst, src, (size_t)bytes);
        return;
    }
    const int64_t pieces = (bytes + IDCOPY_GRAIN_BYTES - 1) / IDCOPY_GRAIN_BYTES;
    h->idcopy.run(pieces, 1, [&](int64_t b, int64_t e) {
        const int64_t o = b * IDCOPY_GRAIN_BYTES;
        const int64_t n = std::min(bytes, e * IDCOPY_GRAIN_BYTES) - o;
        memcpy((char *)dst + o, (const char *)src + o, (size_t)n);
    });
}

// `ahead`: the batch is only prepared, held by a later plan (window index
// above the lookahead).  Its arrays in the caller's device memory may be read
// after this sp_plan call returns: the query of the first plan that holds the
// batch waits for this ingest, and that plan waits for the query.
// `prestaged`: a batch from host memory already copied into the entry's
// pinned buffers (by defer_ahead).
static sp_status ingest(sp_ctx *h, const sp_batch &bt, int64_t q, bool ahead,
                        bool prestaged = false)
{
    const int r = (int)(q % h->nring);
    BatchDev &b = h->ring[r];
    hipStream_t si = h->s_ingest;
    // this call returns only once the caller's device arrays have been read
    const bool caller_waits = bt.on_device && !ahead;
    // the previous occupant (batch q - nring) must be done with its backward
    HIPCHK(h, wait_unless_done(si, h->ev_upd[r]));
    // With the staged fill the step is bound by the host's gather, and a batch
    // sorted ahead has time to spare: it waits for the last update issued, so
    // that the training kernels do not share the GPU with it.  Not one the
    // host waits for.
    if (h->staged && h->updated > 0 && !caller_waits)
        HIPCHK(h, wait_unless_done(si, h->ev_upd[(h->updated - 1) % h->nring]));
    const bool timing = h->flags & SP_FLAG_TIMING;
    if (timing) HIPCHK(h, h->t_ing.begin(si));
    const int64_t nbags = (int64_t)h->T * bt.batch;
    const int32_t *ids = bt.ids, *off = bt.bag_off;
    if (!bt.on_device) {
        // host arrays: copied on the host into this entry's pinned buffers
        // (the caller's arrays are free again right after), then to the ring
        // asynchronously.  The buffers' previous copy (batch q - nring, or
        // this batch before a rejected plan) has long run.
        if (!prestaged) {
            if (h->ids_pending[r]) HIPCHK(h, hipEventSynchronize(h->ev_ids[r]));
            copy_host(h, h->h_ids[r], bt.ids, (int64_t)sizeof(int32_t) * bt.nnz);
            memcpy(h->h_off[r], bt.bag_off, sizeof(int32_t) * (nbags + 1));
        }
        if (bt.nnz > 0)
            HIPCHK(h, hipMemcpyAsync(b.ids, h->h_ids[r], sizeof(int32_t) * bt.nnz,
                                     hipMemcpyHostToDevice, si));
        HIPCHK(h, hipMemcpyAsync(b.bag_off, h->h_off[r], sizeof(int32_t) * (nbags + 1),
                                 hipMemcpyHostToDevice, si));
        HIPCHK(h, hipEventRecord(h->ev_ids[r], si));
        h->ids_pending[r] = 1;
        ids = b.ids;
        off = b.bag_off;
    }
    IngestCons ic{h->cons_counter, 0, h->h_cnt_dev + COUNTER_WORDS, 0};
    if (bt.nnz > 0 && ingest_in_lds(h->max_table_ids, bt.batch)) {
        // one launch; it reports when it has read its inputs, which matters
        // only for the caller's device arrays
        h->cons_issued += (uint32_t)(h->T * ingest_splits(h->T));
        ic.target = h->cons_issued;
        ic.seq = ++h->cons_seq;
        if (caller_waits) {
            h->wait_cons_word = true;
            h->wait_seq = ic.seq;
        }
    } else if (caller_waits) {
        h->wait_cons_event = true;  // recorded by launch_ingest once the inputs are read
    }
    launch_ingest(h->tb, b, ids, off, bt.batch, bt.nnz, h->key_bits, h->chunk, h->max_table_ids,
                  h->max_ids, h->nchunk_max, h->itmp_k, h->itmp_v, h->ihist, h->ws_ingest,
                  caller_waits ? h->ev_consumed : nullptr, ic, si);
    CHECK_LAUNCH(h);
    if (h->ws_ingest.overflow) return fail(h, SP_ERR_HIP, "internal: scan workspace too small");
    HIPCHK(h, hipEventRecord(h->ring_ready[r], si));
    if (timing) HIPCHK(h, h->t_ing.end(si));
    h->ring_seen[r] = 0;
    h->ring_batch[r] = q;
    h->ring_nnz[r] = bt.nnz;
    h->ring_B[r] = bt.batch;
    return SP_OK;
}

// Issue the pending write-back copy (plan p = copy_pending) on stream s and
// hand its rows to the write-back thread.  The host staging slot was last
// used by plan p - nstage, whose scatter is joined first.
static sp_status issue_copy(sp_ctx *h, hipStream_t s)
{
    const int64_t p = h->copy_pending;
    if (p < 0) return SP_OK;
    const int sl = (int)(p % h->nstage);
    TRY(join_fill(h, p));  // ev_filled of plan p is recorded
    if (p >= h->nstage) TRY(join_jobs(h, p - h->nstage));
    Job job;
    job.ticket = p;
    const int64_t n = h->copy_n;
    if (n > 0) {
        HIPCHK(h, wait_unless_done(s, h->ev_filled[p % h->nring]));
        // in pieces: the runtime copies device to host with a blit kernel
        // that keeps a workgroup on every compute unit until it ends, and
        // one copy of a large write-back runs for most of the step; pieces
        // end often enough for the training kernels' workgroups to take
        // those units (the 26x10M update: 0.63 ms beside pieces of 32 MiB,
        // 0.74-0.84 ms beside one copy of 911 MB)
        const int64_t bytes = (int64_t)sizeof(float) * n * (h->D + 1);
        for (int64_t off = 0; off < bytes; off += WB_PIECE_BYTES)
            HIPCHK(h, hipMemcpyAsync((char *)h->stage_host[sl] + off,
                                     (const char *)h->stage_dev[sl] + off,
                                     std::min(WB_PIECE_BYTES, bytes - off),
                                     hipMemcpyDeviceToHost, s));
        HIPCHK(h, hipEventRecord(h->ev_d2h[sl], s));
        job.ev = h->ev_d2h[sl];
        job.rows = h->stage_host[sl];
        job.keys = (const int32_t *)(h->stage_host[sl] + n * h->D);
        job.n = n;
    }
    {
        std::lock_guard<std::mutex> lk(h->mu);
        h->jobs.push_back(job);
    }
    h->cv.notify_one();
    h->copy_pending = -1;
    return SP_OK;
}

// Ingest the window's batches after the hold window (prepared ahead) that are
// not in the ring yet.
static sp_status ingest_ahead(sp_ctx *h, const sp_batch *window, int n, int nhold, int64_t k)
{
    for (int w = nhold; w < n; ++w)
        if (h->ring_batch[(k + w) % h->nring] != k + w) TRY(ingest(h, window[w], k + w, true));
    return SP_OK;
}

// Staged fill with a large write-back copy on the ingest stream: sorted behind
// that copy, the batches prepared ahead would run as the step's training
// kernels do.  Those that no query of this call or the next needs (window
// index above lookahead + 1) are sorted behind the update of this plan's
// ticket instead, where the step waits for the host's gather.  Host arrays
// are copied into the entry's pinned buffers now (the caller's are free when
// sp_plan returns); device ones are read then, before any plan that holds
// them.
static sp_status defer_ahead(sp_ctx *h, const sp_batch *window, int n, int from, int64_t k)
{
    for (int w = from; w < n; ++w) {
        const sp_batch &bt = window[w];
        const int64_t q = k + w;
        const int r = (int)(q % h->nring);
        if (h->ring_batch[r] == q) continue;
        if (!bt.on_device) {
            if (h->ids_pending[r]) HIPCHK(h, hipEventSynchronize(h->ev_ids[r]));
            h->ids_pending[r] = 0;
            copy_host(h, h->h_ids[r], bt.ids, (int64_t)sizeof(int32_t) * bt.nnz);
            memcpy(h->h_off[r], bt.bag_off,
                   sizeof(int32_t) * ((int64_t)h->T * bt.batch + 1));
        }
        h->deferred.push_back({bt, q});
    }
    return SP_OK;
}

// Enqueue the deferred ingests (behind the last update issued).
static sp_status ingest_deferred(sp_ctx *h)
{
    const double t0 = host_ms();
    for (const auto &d : h->deferred) TRY(ingest(h, d.bt, d.q, true, !d.bt.on_device));
    h->deferred.clear();
    h->host_ms[0] += host_ms() - t0;
    return SP_OK;
}

// RAW-4: a row evicted by plan p may be refilled from plan p + n_p on (n_p
// batches in p's hold window; n_p - d with prefetch depth d, which fills the
// batches after the planned one): before plan k reads the host tables for
// its fill, every write-back due by then has landed.
static sp_status join_writebacks(sp_ctx *h, int64_t k)
{
    int64_t need = -1;
    for (const auto &d : h->deadlines)
        if (d.second <= k) need = std::max(need, d.first);
    if (need >= 0) {
        if (h->copy_pending >= 0 && h->copy_pending <= need) TRY(issue_copy(h, h->s_copy));
        TRY(join_jobs(h, need));
        while (!h->deadlines.empty() && h->deadlines.front().first <= need) h->deadlines.pop_front();
    }
    return SP_OK;
}

// Wait until the ingests of held batches that this sp_plan call enqueued have
// read the caller's device arrays: the general path's event, and the word an
// ingest in LDS writes once its blocks have read their inputs (stream order
// makes the last one enough).  After a query this returns at once: the query
// waited for those ingests.  Stream errors end the wait; they surface on the
// next call that checks the stream.
static void wait_inputs_read(sp_ctx *h)
{
    const double t0 = host_ms();
    if (h->wait_cons_event) (void)hipEventSynchronize(h->ev_consumed);
    if (h->wait_cons_word) {
        const volatile uint64_t *w = h->h_cnt + COUNTER_WORDS;
        // words arrive in stream order; a later ingest's may already be there
        for (int64_t spin = 0; (int32_t)((uint32_t)*w - h->wait_seq) < 0; ++spin) {
            if ((spin & 1023) == 1023 && hipStreamQuery(h->s_ingest) != hipErrorNotReady) {
                (void)hipGetLastError();
                break;  // idle (the word is final) or failed
            }
            __builtin_ia32_pause();
        }
    }
    h->wait_cons_event = h->wait_cons_word = false;
    h->host_ms[5] += host_ms() - t0;
}

// Wait until the query with sequence number seq has published every counter
// word, and copy them out.  The host polls the coherent words instead of
// synchronising the stream: the values count, not the end of the kernel, and
// the plan stream keeps its order for what comes next.  Stream errors end the
// wait.
static sp_status wait_counts(sp_ctx *h, uint32_t seq, DevCounters *c)
{
    int32_t *dst = reinterpret_cast<int32_t *>(c);
    const volatile uint64_t *w = h->h_cnt;
    for (int64_t spin = 0;; ++spin) {
        bool all = true;
        for (int i = 0; i < COUNTER_WORDS && all; ++i) {
            const uint64_t x = w[i];
            all = (uint32_t)(x >> 32) == seq;
            dst[i] = (int32_t)(uint32_t)x;
        }
        if (all) return SP_OK;
        if ((spin & 1023) == 1023) {
            const hipError_t e = hipStreamQuery(h->s_plan);
            if (e == hipSuccess) {  // the stream is idle, so the words are final
                for (int i = 0; i < COUNTER_WORDS; ++i) {
                    const uint64_t x = w[i];
                    if ((uint32_t)(x >> 32) != seq)
                        return fail(h, SP_ERR_HIP, "internal: plan counters were not published");
                    dst[i] = (int32_t)(uint32_t)x;
                }
                return SP_OK;
            }
            if (e != hipErrorNotReady) {
                (void)hipGetLastError();
                return fail(h, SP_ERR_HIP, "plan stream: %s", hipGetErrorString(e));
            }
        }
        __builtin_ia32_pause();
    }
}

// Phase 1 of plan k over window batches k .. k+nhold-1, all ingested or being
// ingested: the planned batch's hits, the stamps of the entering batches'
// cached slots, and per-table miss / held counts, published to host-coherent
// memory (Storage, the Hit-Map and the holds are not written).
static sp_status enqueue_query(sp_ctx *h, int64_t k, int nhold, uint32_t *seq_out)
{
    const int e = (int)(k % h->nring);
    const bool timing = h->flags & SP_FLAG_TIMING;
    if (timing) HIPCHK(h, h->t_qry.begin(h->s_plan));
    // the ticket buffers being reused belonged to ticket k - nring
    if (k >= h->nring) HIPCHK(h, wait_unless_done(h->s_plan, h->ev_upd[e]));
    TicketHost &th = h->tkh[e];
    int64_t nnz[MAX_WINDOW] = {};
    for (int w = 0; w < nhold; ++w) {
        const int r = (int)((k + w) % h->nring);
        if (!h->ring_seen[r]) {  // later queries are behind this one on the same stream
            HIPCHK(h, wait_unless_done(h->s_plan, h->ring_ready[r]));
            h->ring_seen[r] = 1;
        }
        th.uk[w] = h->ring[r].ukeys;
        th.nu[w] = h->ring[r].scal;
        nnz[w] = h->ring_nnz[r];
    }
    // the past window: batches planned before k stay in the ring (nring covers them)
    int nwin = nhold;
    for (int64_t q = k - 1; q >= 0 && q >= k - h->P; --q, ++nwin) {
        const int r = (int)(q % h->nring);
        if (h->ring_batch[r] != q)
            return fail(h, SP_ERR_HIP, "internal: past batch %lld is not in the window ring", (long long)q);
        th.uk[nwin] = h->ring[r].ukeys;
        th.nu[nwin] = h->ring[r].scal;
        nnz[nwin] = h->ring_nnz[r];
    }
    const PrefetchDev pf{std::min(h->pf_depth, nhold - 1), h->pf_own_key, h->pf_own_uidx,
                         h->pf_flag, h->max_ids};
    // rows: the planned batch, the successors to prefetch, and the batches
    // entering the hold window.  A batch marked held by an earlier plan but no
    // longer in the window (the caller shortened it) makes every hold be
    // rebuilt from this window and the past ones.
    QueryRows &qr = th.qr;
    qr = QueryRows{};
    qr.span = h->L + h->P;
    qr.rebuild = h->entered > k + nhold - 1;
    int64_t max_nnz = 0;
    for (int w = 0; w < nwin; ++w) {
        qr.qoff[w] = w < nhold ? w : -(w - nhold + 1);
        qr.eslot[w] = h->ring[(k + qr.qoff[w]) % h->nring].eslot;
        th.ent_len[w] = nnz[w];
        const bool ent = qr.rebuild || (w < nhold && k + w > h->entered);
        if (ent) qr.entrant |= 1u << w;
        if (w == 0 || w <= pf.depth || ent) {
            qr.idx[qr.n++] = w;
            max_nnz = std::max(max_nnz, nnz[w]);
        }
    }
    th.stamp = ++h->stamp;
    *seq_out = ++h->qseq;
    // Staged fill without prefetch, while plans write rows back: the query
    // itself hands the missing keys to the host (their pinned slot was last
    // read by the gather of plan k - nstage), so the gather needs no copy
    // first.  Its stores to host memory are slow, though, and the counts it
    // publishes last arrive behind them: when nothing is written back (the
    // step then waits on the counts, not on the host link) the plan copies
    // the keys instead.  Measured: 26x10M 1.2% faster with the stores, the
    // mixed workload 17% faster with the copy.
    const int sl = (int)(k % h->nstage);
    uint32_t *host_keys = nullptr;
    th.keys_direct = h->staged && pf.depth == 0 && !h->last_fresh;
    if (th.keys_direct) {
        TRY(join_fill(h, k - h->nstage));
        host_keys = h->h_mkey_dev[sl];
    }
    launch_query(h->tb, h->hash, h->hash_mask, th.uk, th.nu, nwin, max_nnz, h->hold_to, h->held,
                 th.stamp, h->hcnt, (int32_t)k, qr, RowIndex{h->rbase, h->lastq, h->pend}, h->tk[e],
                 pf, h->cnt, h->cnt_part,
                 h->cnt_part + PART_COPIES * PART_WORDS, h->ring[k % h->nring].scal, h->h_cnt_dev,
                 *seq_out, host_keys, h->stage_rows, h->ws_plan, h->s_plan);
    CHECK_LAUNCH(h);
    if (host_keys) HIPCHK(h, hipEventRecord(h->ev_mkey[sl], h->s_plan));  // the keys are complete
    if (h->ws_plan.overflow) return fail(h, SP_ERR_HIP, "internal: scan workspace too small");
    if (timing) HIPCHK(h, h->t_qry.end(h->s_plan));
    return SP_OK;
}

extern "C" sp_status sp_plan(sp_handle h, const sp_batch *window, int32_t n, int64_t *ticket)
{
    TRY(usable(h));
    if (h->updated != h->planned)
        return fail(h, SP_ERR_SEQUENCE, "plan %lld requested before backward of ticket %lld",
                    (long long)h->planned, (long long)h->planned - 1);
    if (!window || n < 1 || n > h->L + 1 + SP_MAX_AHEAD)
        return fail(h, SP_ERR_INVALID_ARG, "window of %d batches (1..%d allowed)", n,
                    h->L + 1 + SP_MAX_AHEAD);
    for (int w = 0; w < n; ++w) {
        const sp_batch &b = window[w];
        if (b.batch < 0 || b.batch > h->max_batch || b.nnz < 0 || b.nnz > h->max_ids || !b.bag_off ||
            (b.nnz > 0 && !b.ids) || (b.batch == 0 && b.nnz != 0))
            return fail(h, SP_ERR_INVALID_ARG, "window[%d]: batch %d / nnz %lld outside the config or null pointer",
                        w, b.batch, (long long)b.nnz);
    }
    // normally enqueued by the last sp_backward_update already
    if (!h->deferred.empty()) TRY(ingest_deferred(h));
    const int64_t k = h->planned;
    const int32_t u = (int32_t)k;
    const int e = (int)(k % h->nring);
    const int nhold = std::min<int>(n, h->L + 1);  // window[L+1..], if given, are only prepared
    TicketDev &tk = h->tk[e];
    TicketHost &th = h->tkh[e];
    const bool timing = h->flags & SP_FLAG_TIMING;

    // ---- ingest (own stream): held batches not in the ring yet (normally
    // none once batches are handed over one step early) go now, before the
    // query that needs them; the prepared-ahead batch goes after the query
    // has been enqueued, so its launches overlap the query on the GPU
    double tA = host_ms();
    struct ConsumedGuard {  // the window buffers are the caller's again when we return
        sp_ctx *h;
        ~ConsumedGuard() { wait_inputs_read(h); }
    } guard{h};
    for (int w = 0; w < n; ++w) {
        const int64_t q = k + w;
        const int r = (int)(q % h->nring);
        if (h->ring_batch[r] == q && (h->ring_nnz[r] != window[w].nnz || h->ring_B[r] != window[w].batch))
            return fail(h, SP_ERR_INVALID_ARG, "batch %lld changed shape between windows", (long long)q);
        if (w < nhold && h->ring_batch[r] != q) {
            TRY(ingest(h, window[w], q, false));
        }
    }

    double tB = host_ms();
    h->host_ms[0] += tB - tA;
    // ---- phase 1: query and hold, unless the previous plan already issued it
    // over this same window (its batches still in place)
    bool spec = h->spec_ticket == k && h->spec_nhold == nhold;
    for (int w = 0; w < nhold && spec; ++w) spec = h->ring_batch[(k + w) % h->nring] == k + w;
    h->spec_ticket = -1;
    uint32_t seq = h->spec_seq;
    if (!spec) TRY(enqueue_query(h, k, nhold, &seq));
    const int r0 = (int)(k % h->nring);
    double tC = host_ms();
    h->host_ms[1] += tC - tB;
    // batches prepared ahead: with the staged fill they wait until the gather
    // has its keys (their host copy would delay it)
    if (!h->staged) TRY(ingest_ahead(h, window, n, nhold, k));
    double tD = host_ms();
    h->host_ms[0] += tD - tC;
    DevCounters c;
    TRY(wait_counts(h, seq, &c));
    double tE = host_ms();
    h->host_ms[2] += tE - tD;
    if (c.err & (ERR_ID_RANGE | ERR_OFFSETS | ERR_TABLE_IDS)) {
        for (int w = 0; w < n; ++w) h->ring_batch[(k + w) % h->nring] = -1;  // re-read on retry
        return fail(h, SP_ERR_INVALID_ARG, "%s in the window",
                    (c.err & ERR_ID_RANGE)  ? "row ID out of range"
                    : (c.err & ERR_OFFSETS) ? "malformed bag offsets"
                                            : "a table with more IDs than max_table_ids");
    }
    if (c.err_sticky)
        return fail(h, SP_ERR_HIP, "internal planner inconsistency (flags %d) in an earlier plan",
                    c.err_sticky);
    // prefetch mode: the successors' rows to fetch count as misses too
    const int pf_d = std::min(h->pf_depth, nhold - 1);
    const bool pf_on = pf_d > 0;
    int32_t pf_tot[MAX_TABLES];
    for (int t = 0; t < h->T; ++t) {
        pf_tot[t] = 0;
        for (int w = 0; w < MAX_PF; ++w) {
            if (w >= pf_d) c.pf[w][t] = 0;
            pf_tot[t] += c.pf[w][t];
        }
    }
    int64_t n_miss = 0, n_own = 0, margin = INT64_MAX;
    for (int t = 0; t < h->T; ++t) {
        const int64_t free_slots = h->slots[t] - c.held[t];
        const int64_t need = (int64_t)c.miss[t] + pf_tot[t];
        margin = std::min<int64_t>(margin, free_slots - need);
        if (need > free_slots) {
            for (int w = 0; w < n; ++w) h->ring_batch[(k + w) % h->nring] = -1;  // re-read on retry
            return fail(h, SP_ERR_CAPACITY,
                        "table %d: %lld misses (%d to prefetch) but only %lld unheld slots (plan %lld)",
                        t, (long long)need, pf_tot[t], (long long)free_slots, (long long)k);
        }
        n_miss += need;
        n_own += c.miss[t];
    }

    // ---- phase 2: commit
    const BatchDev &b0 = h->ring[r0];
    th.nnz = h->ring_nnz[r0];
    th.B = (int32_t)h->ring_B[r0];
    th.n_unique = c.n_unique;
    th.n_chunks = c.n_chunks;
    th.n_multi = c.n_multi;
    th.n_miss = n_miss;
    th.n_own = n_own;
    th.ring = r0;
    th.nwin = nhold;

    if (pf_on && n_miss > 0) {
        // the miss list: per table own misses, then each successor's rows to
        // prefetch (the query left the own misses aside); it needs only the
        // query's outputs and counts, not the victims
        const int32_t *n_next[MAX_PF] = {};
        const uint32_t *next_keys[MAX_PF] = {};
        int64_t max_next[MAX_PF] = {};
        for (int w = 0; w < pf_d; ++w) {
            const int r1 = (int)((k + 1 + w) % h->nring);
            n_next[w] = h->ring[r1].scal;
            next_keys[w] = h->ring[r1].ukeys;
            max_next[w] = h->ring_nnz[r1];
        }
        launch_pf_arrange(h->tb,
                          PrefetchDev{pf_d, h->pf_own_key, h->pf_own_uidx, h->pf_flag, h->max_ids},
                          n_own, n_next, max_next, next_keys, c.miss, c.pf, tk, n_miss,
                          &h->cnt->err_sticky, h->ws_plan, h->s_plan);
    }
    if (h->staged && n_miss > 0) {
        // the staged fill gathers on the host as soon as it has the missing
        // keys, while the victims are chosen: they go first.  Their pinned
        // slot was last read by the fill of plan k - nstage.  ev_mkey marks
        // them complete.
        const int sl = (int)(k % h->nstage);
        if (!th.keys_direct) {  // (otherwise the query wrote them there itself)
            TRY(join_fill(h, k - h->nstage));
            HIPCHK(h, hipMemcpyAsync(h->h_mkey[sl], tk.m_key, sizeof(uint32_t) * n_miss,
                                     hipMemcpyDeviceToHost, h->s_plan));
            HIPCHK(h, hipEventRecord(h->ev_mkey[sl], h->s_plan));
        }
        // the gather reads the host tables: the write-backs due land first
        TRY(join_writebacks(h, k));
        MoveJob gj;
        gj.gather = true;
        gj.k = k;
        gj.n = n_miss;
        gj.sl = sl;
        gj.timing = timing;
        {
            std::lock_guard<std::mutex> lk(h->fmu);
            h->fjobs.push_back(gj);
        }
        h->fcv.notify_one();
        // The victims and the commit are then off the step's path (the gather
        // takes far longer): they wait for the update of the batch before,
        // so that the training kernels do not share the GPU with them.
        if (k >= 1) HIPCHK(h, wait_unless_done(h->s_plan, h->ev_upd[(k - 1) % h->nring]));
    }
    if (timing) HIPCHK(h, h->t_plan.begin(h->s_plan));
    // the plan is accepted: the entering batches' cached slots become held.
    // The commit marks them (the victims are chosen without them: the query
    // stamped them); a rebuild drops every hold and marks them first.
    HoldRows hr{};
    for (int r = 0; r < th.qr.n; ++r) {
        const int w = th.qr.idx[r];
        if (!((th.qr.entrant >> w) & 1u)) continue;
        const int y = hr.n++;
        hr.uk[y] = th.uk[w];
        hr.nu[y] = th.nu[w];
        hr.es[y] = th.qr.eslot[w];
        hr.nv_off[y] = th.qr.qoff[w] + h->P;
        hr.q_off[y] = th.qr.qoff[w];
        hr.start[y + 1] = hr.start[y] + th.ent_len[w];
    }
    const RowIndex ri{h->rbase, h->lastq, h->pend};
    // the filled rows' holds from lastq / pend when at most one batch enters
    const bool fast_hold = !th.qr.rebuild && hr.n <= 1;
    const int32_t ent = hr.n == 1 ? hr.q_off[0] : 0;
    if (th.qr.rebuild) {
        launch_hold_rebuild(h->tb, hr, ri, h->hold_to, h->hcnt, u, h->s_plan);
        hr = HoldRows{};
    }

    if (n_miss > 0) {
        const int64_t cap = (int64_t)h->hash_mask + 1;
        if (h->hash_used + n_miss > cap * 7 / 10) {
            launch_hash_rebuild(h->hash, h->hash_mask, h->key_of_slot, h->total_slots, h->cnt, h->s_plan);
            h->hash_used = h->total_slots;
            ++h->st.hash_rebuilds;
        }
        h->hash_used += n_miss;
        // every table's victims among its never-used slots: no select (with
        // LFU and prefetch never-used slots are not known to come first)
        bool fresh = !(h->policy == POLICY_LFU && pf_on);
        for (int t = 0; t < h->T; ++t)
            fresh = fresh && c.miss[t] + pf_tot[t] <= h->slots[t] - h->fresh[t];
        SelArgs a{};
        FreshArgs f{};
        int32_t vb = 0;
        int64_t maxS = 0, maxK = 0;
        for (int t = 0; t < h->T; ++t) {
            const int64_t kt = c.miss[t] + pf_tot[t];
            if (fresh && kt > 0) {
                const int y = f.n++;
                f.vbase[y] = vb;
                f.k[y] = (int32_t)kt;
                f.first[y] = h->tb.slot_base[t] + h->fresh[t];
                maxK = std::max(maxK, kt);
            } else if (kt > 0) {
                int y = a.nact++;
                a.t[y] = t;
                a.k[y] = c.miss[t] + pf_tot[t];
                a.base[y] = h->tb.slot_base[t];
                a.S[y] = h->slots[t];
                a.vbase[y] = vb;
                maxS = std::max<int64_t>(maxS, h->slots[t]);
            }
            vb += c.miss[t] + pf_tot[t];
            // the first kt never-used slots are taken either way (all of them
            // when there are fewer)
            h->fresh[t] = std::min<int64_t>(h->slots[t], h->fresh[t] + kt);
        }
        h->last_fresh = fresh;
        // priority values: LRU last use + 1 <= u, LFU uses <= u + 1, random <= 2^24
        const int nb = h->policy == POLICY_RANDOM ? 25
                       : std::max(1, bits_for((uint64_t)u + (h->policy == POLICY_LFU)));
        a.prio_bits = nb;
        a.act_bits = bits_for((uint64_t)(a.nact - 1));
        a.plan = u;
        a.stamp = th.stamp;
        a.prio = Prio{h->policy == POLICY_LFU ? h->uses : h->last_use, h->policy, (uint32_t)u, h->seed};
        const int levels = (nb + SEL_BITS - 1) / SEL_BITS;
        if (fresh)
            launch_fresh_victims(f, maxK, tk.v_slot, h->s_plan);
        else
            launch_select_victims(a, levels, maxS, h->hold_to, h->held, h->sel_state, h->sel_hist, h->vk0,
                                  h->vv0, h->vk1, (uint32_t *)nullptr, n_miss, h->hist,
                                  h->ws_plan, tk.v_slot, &h->cnt->err_sticky, h->s_plan);
    }
    WindowKeys wk{};
    wk.n = nhold;
    wk.hold_past = h->P;
    wk.fast = fast_hold;
    wk.ent = ent;
    wk.stamp = th.stamp;
    for (int w = 0; w < nhold; ++w) wk.uk[w] = th.uk[w], wk.nu[w] = th.nu[w];
    launch_commit(h->tb, h->hash, h->hash_mask, tk, b0, n_miss, th.n_unique, th.nnz, h->key_of_slot,
                  h->last_use, h->uses, u, pf_on, wk, hr, ri, h->hold_to, h->hcnt, h->cnt, h->s_plan);
    CHECK_LAUNCH(h);
    h->entered = th.qr.rebuild ? k + nhold - 1 : std::max(h->entered, k + nhold - 1);
    if (h->ws_plan.overflow) return fail(h, SP_ERR_HIP, "internal: scan workspace too small");
    HIPCHK(h, hipStreamWriteValue64(h->s_plan, h->sem + SEM_PLANNED, (uint64_t)k + 1, 0));
    // the event only serves event-wait mode; value waits on SEM_PLANNED always work
    th.ev_planned = (h->flags & SP_FLAG_EVENT_WAITS) != 0;
    if (th.ev_planned) HIPCHK(h, hipEventRecord(h->ev_planned[e], h->s_plan));
    if (timing) HIPCHK(h, h->t_plan.end(h->s_plan));
    // a large write-back copy of the previous plan goes on the ingest stream
    // behind this call's ingests (its fill has normally finished by now): it
    // then overlaps this plan's fill (the two use the host link in opposite
    // directions) and is well under way when the next call's ingest comes
    const int64_t copy_bytes = h->copy_pending >= 0 ? h->copy_n * (h->D + 1) * (int64_t)sizeof(float) : 0;
    if (copy_bytes > SMALL_COPY_BYTES) TRY(issue_copy(h, h->s_ingest));
    // With the staged fill the batches prepared ahead are ingested behind that
    // copy on the ingest stream: here only the one the next plan's query holds
    // (normally in the ring already), the rest at the end of this call, where
    // the host's copy of the caller's arrays overlaps that query.
    if (h->staged) TRY(ingest_ahead(h, window, std::min(n, nhold + 1), nhold, k));
    double tF = host_ms();
    h->host_ms[3] += tF - tE;
    // ---- the next plan's query, when its whole window is known: batches
    // k+1 .. k+L+1 are all in the ring now; it runs right behind this commit
    if (n >= h->L + 2) {
        TRY(enqueue_query(h, k + 1, h->L + 1, &h->spec_seq));
        h->spec_ticket = k + 1;
        h->spec_nhold = h->L + 1;
    }
    const double tG = host_ms();
    h->host_ms[1] += tG - tF;
    tF = tG;
    // ---- mover (own stream): write-back of evicted rows and fill of misses;
    // the next plan's query does not wait for it
    if (!h->staged) TRY(join_writebacks(h, k));  // the staged fill joined before its gather
    const int sl = (int)(k % h->nstage);
    MoveJob mj;
    mj.k = k;
    mj.n = n_miss;
    mj.sl = sl;
    mj.e = e;
    mj.u = u;
    mj.timing = timing;
    // the device staging slot is free once plan k - nstage's copy has run
    // (issued two plans ago)
    if (k >= h->nstage && hipEventQuery(h->ev_d2h[sl]) != hipSuccess) {
        (void)hipGetLastError();
        mj.wait[mj.nwait++].ev = h->ev_d2h[sl];
    }
    if (th.ev_planned) {
        mj.wait[mj.nwait++].ev = h->ev_planned[e];
    } else {
        Wait &w = mj.wait[mj.nwait++];
        w.addr = h->sem + SEM_PLANNED;
        w.val = (uint64_t)k + 1;
    }
    if (n_miss > 0) {
        // RAW-2/3: a victim's row is final once the last update that used it
        // has run.  Update j freed ring entry j % nring for batch j + nring,
        // whose ingest waited for it; this plan's query is behind every batch
        // up to k+L, so updates up to k+L-nring are behind this stream
        // already.  Batches k-P .. k-1 of the past window cannot have used a
        // victim's row (their rows are held), and the fill writes only victim
        // slots, so their updates need no wait.  The rest are waited for, one
        // wait when they share a stream.
        // (a value wait: a wait on a pending event costs the host far more)
        const int64_t last = k - 1 - h->P;
        for (int64_t j = std::max<int64_t>(0, k + h->L + 1 - h->nring); j <= last; ++j) {
            const int ej = (int)(j % h->nring);
            if (j != last && h->upd_stream[ej] == h->upd_stream[last % h->nring]) continue;
            if (hipEventQuery(h->ev_upd[ej]) == hipSuccess) continue;  // already done
            (void)hipGetLastError();
            if (mj.nwait == (int)(sizeof mj.wait / sizeof mj.wait[0]))
                return fail(h, SP_ERR_HIP, "internal: too many waits for the fill");
            Wait &w = mj.wait[mj.nwait++];
            if (!h->upd_val[ej]) {  // that update wrote no word (event-wait mode then)
                w.ev = h->ev_upd[ej];
            } else {
                w.addr = h->sem + SEM_UPD + 8 * ej;
                w.val = (uint64_t)j + 1;
            }
        }
    }
    if (h->staged) {
        {
            std::lock_guard<std::mutex> lk(h->fmu);
            h->fjobs.push_back(mj);
        }
        h->fcv.notify_one();
    } else {
        HIPCHK(h, enqueue_move(h, mj, nullptr));
    }
    // a small one goes on the copy stream now: it ends long before the next
    // fill, even where its queue is the move stream's
    TRY(issue_copy(h, h->s_copy));
    h->copy_pending = k;
    h->copy_n = n_miss;
    // an evicted row is in no batch of this plan's window, so the first plan
    // that can fill it again is the one whose planned batch (or, prefetching,
    // next batch) is the first after the window
    h->deadlines.emplace_back(k, k + nhold - pf_d);

    h->host_ms[4] += host_ms() - tF;
    h->planned = k + 1;
    h->st.plans += 1;
    h->st.lookups += th.nnz;
    h->st.unique += th.n_unique;
    h->st.misses += n_miss;
    h->st.hits += th.n_unique - n_own;
    h->st.prefetched += n_miss - n_own;
    h->st.bytes_fill += n_miss * h->D * (int64_t)sizeof(float);
    h->st.min_capacity_margin = std::min(h->st.min_capacity_margin, margin);
    if (ticket) *ticket = k;
    if (h->staged) {
        const double t0 = host_ms();
        if (copy_bytes > DEFER_BEHIND_COPY_BYTES || (h->flags & SP_FLAG_DEFER_SORTS))
            TRY(defer_ahead(h, window, n, nhold + 1, k));
        else
            TRY(ingest_ahead(h, window, n, nhold, k));
        h->host_ms[0] += host_ms() - t0;
    }
    if (h->flags & SP_FLAG_DEBUG_SYNC) HIPCHK(h, hipDeviceSynchronize());
    return SP_OK;
}

// ---------------------------------------------------------------- forward / backward

extern "C" sp_status sp_forward(sp_handle h, int64_t ticket, float *d_out, void *stream)
{
    TRY(usable(h));
    if (ticket != h->planned - 1 || h->forwarded != ticket)
        return fail(h, SP_ERR_SEQUENCE, "forward of ticket %lld out of order (planned %lld, forwarded %lld)",
                    (long long)ticket, (long long)h->planned, (long long)h->forwarded);
    const int e = (int)(ticket % h->nring);
    const TicketHost &th = h->tkh[e];
    const int64_t nbags = (int64_t)h->T * th.B;
    if (nbags > 0 && !d_out) return fail(h, SP_ERR_INVALID_ARG, "null d_out");
    hipStream_t s = (hipStream_t)stream;
    // The batch's rows are resident once the fills that brought them are done:
    // this plan's, if the batch had misses of its own (its fill also follows
    // the commit that wrote slot_of); otherwise earlier ones only (with
    // prefetch the previous plan's), and the commit is waited for by itself.
    // This plan's fill writes only victim slots, which hold no row of the
    // batch, so the forward and the update then overlap it.
    const bool ev = h->flags & SP_FLAG_EVENT_WAITS;
    // staged fill: the fill waited for must be enqueued before anything waits on it
    TRY(join_fill(h, th.n_own > 0 || ticket == 0 ? ticket : ticket - 1));
    if (th.n_own > 0 || ticket == 0) {
        if (ev) HIPCHK(h, hipStreamWaitEvent(s, h->ev_filled[e], 0));
        else HIPCHK(h, hipStreamWaitValue64(s, h->sem + SEM_FILLED, (uint64_t)ticket + 1,
                                            hipStreamWaitValueGte, ~0ull));
    } else {
        if (ev && th.ev_planned) {
            HIPCHK(h, hipStreamWaitEvent(s, h->ev_planned[e], 0));
            HIPCHK(h, hipStreamWaitEvent(s, h->ev_filled[(ticket - 1) % h->nring], 0));
        } else {
            HIPCHK(h, hipStreamWaitValue64(s, h->sem + SEM_PLANNED, (uint64_t)ticket + 1,
                                           hipStreamWaitValueGte, ~0ull));
            HIPCHK(h, hipStreamWaitValue64(s, h->sem + SEM_FILLED, (uint64_t)ticket,
                                           hipStreamWaitValueGte, ~0ull));
        }
    }
    // RAW-1: the previous update must land first (implicit on the same stream)
    if (ticket >= 1 && s != h->last_update_stream)
        HIPCHK(h, wait_unless_done(s, h->ev_upd[(ticket - 1) % h->nring]));
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if ((h->flags & SP_FLAG_TIMING) && nbags > 0) HIPCHK(h, h->t_fwd.take(&e0, &e1));
    launch_forward(h->storage, h->D, h->total_slots, h->tk[e].slot_of, h->ring[th.ring].bag_off,
                   nbags, d_out, s, e0, e1);
    CHECK_LAUNCH(h);
    h->forwarded = ticket + 1;
    if (h->flags & SP_FLAG_DEBUG_SYNC) HIPCHK(h, hipDeviceSynchronize());
    return SP_OK;
}

// Backward and update of a ticket, the split runs' partial sums in `partial`
// (the context's buffer, or the fixed array of the static entry point, which
// holds at most partial_bytes).  `defer`: then enqueue the ingests that
// sp_plan deferred (the static entry point leaves them to the next sp_plan and
// enqueues nothing on the library's streams).
static sp_status backward_update(sp_handle h, int64_t ticket, const float *d_grad, float lr,
                                 void *stream, float *partial, int64_t partial_bytes, bool defer)
{
    TRY(usable(h));
    if (ticket != h->forwarded - 1 || h->updated != ticket)
        return fail(h, SP_ERR_SEQUENCE, "backward of ticket %lld out of order (forwarded %lld, updated %lld)",
                    (long long)ticket, (long long)h->forwarded, (long long)h->updated);
    const int e = (int)(ticket % h->nring);
    const TicketHost &th = h->tkh[e];
    if (th.nnz > 0 && !d_grad) return fail(h, SP_ERR_INVALID_ARG, "null d_grad");
    // partials are indexed by chunk: room for every chunk of the ticket
    if (th.n_multi > 0 && th.n_chunks * h->D * (int64_t)sizeof(float) > partial_bytes)
        return fail(h, SP_ERR_INVALID_ARG,
                    "ticket %lld has %lld backward chunks of %d floats: %lld bytes of partial sums, "
                    "above the %lld available",
                    (long long)ticket, (long long)th.n_chunks, h->D,
                    (long long)(th.n_chunks * h->D * (int64_t)sizeof(float)), (long long)partial_bytes);
    hipStream_t s = (hipStream_t)stream;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    if ((h->flags & SP_FLAG_TIMING) && th.n_chunks > 0) HIPCHK(h, h->t_bwd.take(&ev[0], &ev[1]));
    if ((h->flags & SP_FLAG_TIMING) && th.n_chunks > 0 && th.n_multi > 0)
        HIPCHK(h, h->t_cmb.take(&ev[2], &ev[3]));
    launch_backward(h->storage, h->D, h->total_slots, h->ring[th.ring], h->tk[e].slot_u,
                    th.n_chunks, th.n_multi, h->chunk, d_grad, (int64_t)h->T * th.B, lr,
                    partial, s, ev);
    CHECK_LAUNCH(h);
    HIPCHK(h, hipEventRecord(h->ev_upd[e], s));  // also frees ring entry e of the window
    h->upd_val[e] = !(h->flags & SP_FLAG_EVENT_WAITS);
    if (h->upd_val[e])  // for the value wait of a later fill
        HIPCHK(h, hipStreamWriteValue64(s, h->sem + SEM_UPD + 8 * e, (uint64_t)ticket + 1, 0));
    h->upd_stream[e] = s;
    h->last_update_stream = s;
    h->updated = ticket + 1;
    h->st.updates += 1;
    h->st.chunks += th.n_chunks;
    if (defer) TRY(ingest_deferred(h));
    if (h->flags & SP_FLAG_DEBUG_SYNC) HIPCHK(h, hipDeviceSynchronize());
    return SP_OK;
}

extern "C" sp_status sp_backward_update(sp_handle h, int64_t ticket, const float *d_grad, float lr,
                                        void *stream)
{
    if (!h) return SP_ERR_STATE;
    return backward_update(h, ticket, d_grad, lr, stream, h->partial,
                           h->nchunk_max * h->D * (int64_t)sizeof(float), true);
}

extern "C" sp_status sp_backward_update_static(sp_handle h, int64_t ticket, const float *d_grad,
                                               float lr, void *stream)
{
    if (!h) return SP_ERR_STATE;
    return backward_update(h, ticket, d_grad, lr, stream, h->static_partial, STATIC_PARTIAL_BYTES,
                           false);
}

// ---------------------------------------------------------------- flush / stats / debug

extern "C" sp_status sp_flush(sp_handle h)
{
    TRY(usable(h));
    TRY(join_fill(h, h->planned - 1));
    TRY(issue_copy(h, h->s_copy));
    HIPCHK(h, hipDeviceSynchronize());
    TRY(join_jobs(h, h->planned - 1));
    h->deadlines.clear();
    std::vector<int32_t> keys((size_t)h->total_slots);
    HIPCHK(h, hipMemcpy(keys.data(), h->key_of_slot, sizeof(int32_t) * h->total_slots,
                        hipMemcpyDeviceToHost));
    const int rb = h->tb.row_bits;
    const uint32_t mask = (1u << rb) - 1u;
    const size_t row_bytes = sizeof(float) * (size_t)h->D;
    for (int64_t s0 = 0; s0 < h->total_slots; s0 += h->stage_rows) {
        const int64_t cnt = std::min(h->stage_rows, h->total_slots - s0);
        bool any = false;
        for (int64_t i = 0; i < cnt && !any; ++i) any = keys[s0 + i] >= 0;
        if (!any) continue;
        HIPCHK(h, hipMemcpy(h->stage_host[0], h->storage + s0 * h->D, row_bytes * cnt,
                            hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < cnt; ++i) {
            const int32_t key = keys[s0 + i];
            if (key < 0) continue;
            memcpy(h->host[key >> rb] + (int64_t)(key & mask) * h->D, h->stage_host[0] + i * h->D,
                   row_bytes);
        }
    }
    return SP_OK;
}

extern "C" sp_status sp_sync(sp_handle h)
{
    TRY(usable(h));
    TRY(join_fill(h, h->planned - 1));
    TRY(issue_copy(h, h->s_copy));
    HIPCHK(h, hipDeviceSynchronize());
    TRY(join_jobs(h, h->planned - 1));
    h->deadlines.clear();  // every write-back has landed
    return SP_OK;
}

extern "C" sp_status sp_set_flags(sp_handle h, uint32_t flags)
{
    TRY(usable(h));
    if (flags & ~SP_FLAGS_ALL) return fail(h, SP_ERR_INVALID_ARG, "unknown flags");
    h->flags = flags;
    return SP_OK;
}

extern "C" sp_status sp_get_stats(sp_handle h, sp_stats *out)
{
    TRY(usable(h));
    if (!out) return fail(h, SP_ERR_INVALID_ARG, "null stats");
    TRY(join_fill(h, h->planned - 1));  // the fill thread's timers and counts are final
    HIPCHK(h, hipDeviceSynchronize());
    HIPCHK(h, h->t_h2d.flush());
    HIPCHK(h, h->t_fwd.flush());
    HIPCHK(h, h->t_bwd.flush());
    HIPCHK(h, h->t_cmb.flush());
    HIPCHK(h, h->t_plan.flush());
    HIPCHK(h, h->t_fill.flush());
    HIPCHK(h, h->t_ing.flush());
    HIPCHK(h, h->t_qry.flush());
    sp_stats s = h->st;
    {
        std::lock_guard<std::mutex> lk(h->mu);
        s.evictions = h->wb_evictions;
        s.bytes_writeback = h->wb_bytes;
    }
    if (s.min_capacity_margin == INT64_MAX) s.min_capacity_margin = -1;
    s.device_bytes = h->dev_bytes;
    s.pinned_bytes = h->pinned_bytes;
    s.ms_forward = h->t_fwd.ms;
    s.ms_backward = h->t_bwd.ms;
    s.ms_combine = h->t_cmb.ms;
    s.ms_plan = h->t_plan.ms;
    s.ms_fill = h->t_fill.ms;
    s.timed_forward = h->t_fwd.count;
    s.timed_backward = h->t_bwd.count;
    s.timed_combine = h->t_cmb.count;
    s.host_ms_ingest = h->host_ms[0];
    s.host_ms_query = h->host_ms[1];
    s.host_ms_wait = h->host_ms[2];
    s.host_ms_commit = h->host_ms[3];
    s.host_ms_mover = h->host_ms[4];
    s.host_ms_inputs = h->host_ms[5];
    s.prefetched = h->st.prefetched;
    s.timed_plan = h->t_plan.count;
    s.timed_fill = h->t_fill.count;
    s.ms_ingest = h->t_ing.ms;
    s.ms_query = h->t_qry.ms;
    s.timed_ingest = h->t_ing.count;
    s.timed_query = h->t_qry.count;
    s.host_ms_gather = h->gather_ms;
    s.host_ms_fill_join = h->fill_join_ms;
    s.ms_h2d = h->t_h2d.ms;
    s.timed_h2d = h->t_h2d.count;
    *out = s;
    return SP_OK;
}

extern "C" sp_status sp_debug_plan(sp_handle h, int64_t ticket, sp_plan_dump *d)
{
    TRY(usable(h));
    if (!d) return fail(h, SP_ERR_INVALID_ARG, "null dump");
    if (ticket != h->planned - 1 || ticket < 0)
        return fail(h, SP_ERR_SEQUENCE, "only the latest plan (%lld) can be dumped", (long long)h->planned - 1);
    HIPCHK(h, hipStreamSynchronize(h->s_plan));
    const TicketHost &th = h->tkh[ticket % h->nring];
    const TicketDev &tk = h->tk[ticket % h->nring];
    const BatchDev &b = h->ring[th.ring];
    const int rb = h->tb.row_bits;
    const uint32_t mask = (1u << rb) - 1u;
    const int64_t nu = th.n_unique, nm = th.n_miss, nnz = th.nnz;
    std::vector<uint32_t> keys((size_t)std::max<int64_t>(nu, nm) + 1);
    std::vector<int32_t> tmp((size_t)std::max<int64_t>(nu, nm) + 1);
    d->n_unique = nu;
    d->n_miss = nm;
    d->nnz = nnz;
    if (nu > 0) {
        HIPCHK(h, hipMemcpy(keys.data(), b.ukeys, sizeof(uint32_t) * nu, hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < nu; ++i) {
            d->u_table[i] = (int32_t)(keys[i] >> rb);
            d->u_row[i] = (int32_t)(keys[i] & mask);
        }
        HIPCHK(h, hipMemcpy(tmp.data(), tk.hit, sizeof(int32_t) * nu, hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < nu; ++i) d->hit[i] = (uint8_t)(tmp[i] != 0);
        HIPCHK(h, hipMemcpy(d->slot_u, tk.slot_u, sizeof(int32_t) * nu, hipMemcpyDeviceToHost));
    }
    if (nnz > 0) {
        HIPCHK(h, hipMemcpy(d->inv, b.inv, sizeof(int32_t) * nnz, hipMemcpyDeviceToHost));
        HIPCHK(h, hipMemcpy(d->slot_of, tk.slot_of, sizeof(int32_t) * nnz, hipMemcpyDeviceToHost));
    }
    int64_t nev = 0;
    if (nm > 0) {
        HIPCHK(h, hipMemcpy(keys.data(), tk.m_key, sizeof(uint32_t) * nm, hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < nm; ++i) {
            d->m_table[i] = (int32_t)(keys[i] >> rb);
            d->m_row[i] = (int32_t)(keys[i] & mask);
        }
        HIPCHK(h, hipMemcpy(d->v_slot, tk.v_slot, sizeof(int32_t) * nm, hipMemcpyDeviceToHost));
        HIPCHK(h, hipMemcpy(tmp.data(), tk.v_old_key, sizeof(int32_t) * nm, hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < nm; ++i) {
            d->v_old_row[i] = tmp[i] < 0 ? -1 : (int32_t)((uint32_t)tmp[i] & mask);
            nev += tmp[i] >= 0;
        }
        HIPCHK(h, hipMemcpy(d->v_old_use, tk.v_old_lu, sizeof(int32_t) * nm, hipMemcpyDeviceToHost));
    }
    d->n_evict = nev;
    return SP_OK;
}
