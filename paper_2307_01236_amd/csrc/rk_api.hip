// rk_api.hip -- the C ABI of librkrotor (declared in include/rk.h).
//
// Host side: argument checks, the per-chain precompute of App. C's derived
// quantities, device buffers, kernel launches and read-back.  No step of the
// dynamic program itself runs here; the fill, the choice recovery and Alg. 3
// all run in the kernels of rk_kernels.hip.
#include <algorithm>
#include <mutex>
#include <new>
#include <vector>

#include "rk_host.h"
#include "rk_internal.h"

using rk::DevChain;
using rk::DINF;

struct rk_chain {
    rk::HostChain h;  // the caller's chain and everything derived from it on the host
    // Options the kernels evaluate (rk::host_run_slots): built with the pruning setting
    // run_prune from version run_version of the host data (bumped when it changes).
    bool prune = true, run_prune = true;
    int64_t host_version = 0, run_version = -1;
    rk::RunSlots run;

    int device = -1;
    void *d_chain = nullptr;  // x | xbar | c1 | need1 | need1max | P | need2 | lb (options: run slots)
    DevChain dc{};

    void *own_ws = nullptr;  // tables owned by the chain (rk_solve)
    size_t own_ws_bytes = 0;
    rk::Tables tb{};         // tables of the last solve (own or caller's)
    hipStream_t stream = nullptr;
    int32_t M = -1, W = 0;
    bool queued = false;

    hipEvent_t ev_fill0 = nullptr, ev_fill1 = nullptr;
    // The last fill went into a graph the caller is capturing: its events are not recorded
    // (an event recorded inside a capture does not follow the graph's replays), reads do
    // not wait, and no fill time is known.
    bool in_caller_graph = false;
    int32_t launches = 0;
    rk::Profiler prof;

    // The fill's launch sequence is captured once into a HIP graph and replayed while the
    // budget, the tables, the stream and the profiling switch stay the same.
    hipStream_t own_stream = nullptr;  // used when the caller passes no stream
    hipGraphExec_t gexec = nullptr;
    int32_t g_M = -1;
    const int32_t *g_tables = nullptr;
    hipStream_t g_stream = nullptr;
    bool g_prof = false;

    rk_op *d_ops = nullptr;  // backtrace output
    int64_t d_ops_cap = 0;
    int64_t fills = 0;           // solves queued so far
    int64_t bt_fill = -1;        // the solve whose schedule d_ops holds
    int64_t bt_res[3] = {0, 0, 0};
    int64_t *d_res = nullptr;
    int16_t *d_argrow = nullptr;
    int32_t d_argrow_cap = 0;
};

// Wait for the last fill queued by the library.  A fill inside the caller's graph runs when
// the caller replays it; the caller synchronizes before reading.
static hipError_t wait_fill(rk_chain *c)
{
    return c->in_caller_graph ? hipSuccess : hipEventSynchronize(c->ev_fill1);
}

namespace {

#define HIPCHK(expr)                                    \
    do {                                                \
        if ((expr) != hipSuccess) return RK_E_DEVICE;   \
    } while (0)

// Runs on the chain's device, restoring the caller's current device afterwards.
struct DeviceScope {
    int prev = -1;
    bool ok = true;
    explicit DeviceScope(rk_chain *c)
    {
        if (hipGetDevice(&prev) != hipSuccess) { ok = false; return; }
        if (c->device < 0) c->device = prev;
        else if (c->device != prev && hipSetDevice(c->device) != hipSuccess) ok = false;
    }
    ~DeviceScope()
    {
        int cur = -1;
        if (ok && hipGetDevice(&cur) == hipSuccess && cur != prev && prev >= 0) (void)hipSetDevice(prev);
    }
};

// Geometry of the two tables for budget M: the left pad covers every shift x_i that can
// still land on a budget column; a larger x_i makes its operand infinite everywhere.
struct Geometry {
    int32_t W, padl, stride;
    int64_t rows;  // span rows + the infinity row
};

int geometry(const rk_chain *c, int32_t M, Geometry *g, size_t *bytes)
{
    if (M < 0 || M > RK_MAX_M) return RK_E_INVAL;
    g->W = M + 1;
    g->padl = rk::round64(std::min<int64_t>(c->h.max_x, g->W));
    g->stride = g->padl + rk::round64(g->W);
    g->rows = rk::n_rows(c->h.L) + 1;
    // Opt, ap and the right operand table; with the saving sweep also H and aq
    const int64_t elems = (c->h.refwd.empty() ? 3 : 5) * rk::table_rows(c->h.L) * (int64_t)g->stride;
    if (elems <= 0 || elems > (int64_t(1) << 40)) return RK_E_NOMEM;
    // the products address each operand block with 32-bit byte offsets from its first row;
    // the widest block spans OFFSET_SPAN_L (L - 1) + OFFSET_SPAN_C rows
    if ((rk::OFFSET_SPAN_L * (int64_t)c->h.L + rk::OFFSET_SPAN_C) * g->stride * 4 >= (int64_t(1) << 31))
        return RK_E_NOMEM;
    *bytes = (size_t)elems * sizeof(int32_t);
    return RK_OK;
}

// First solve on a device (or the first after the pruning switch changed): upload the
// derived arrays; create the events and streams once.
int ensure_device(rk_chain *c)
{
    if (c->d_chain && c->run_prune == c->prune && c->run_version == c->host_version) return RK_OK;
    if (c->d_chain) {  // rebuild: the captured launch sequence holds the old arrays
        if (c->queued) HIPCHK(wait_fill(c));
        HIPCHK(hipFree(c->d_chain));
        c->d_chain = nullptr;
        if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
        c->gexec = nullptr;
        c->queued = false;
        c->bt_fill = -1;
    }
    if (!c->h.refwd.empty() && c->h.msaH.size() != c->h.msa.size()) return RK_E_INTERNAL;  // sizes H's launches
    rk::host_run_slots(c->h, c->prune, c->run);
    c->run_prune = c->prune;
    c->run_version = c->host_version;
    const int32_t L = c->h.L, K = c->run.k_run;
    const bool sweep = !c->h.refwd.empty();
    const size_t nx = L + 1, nk = (size_t)L * K, nl = (size_t)L * L, nr = (size_t)rk::n_rows(L);
    const size_t total = nx + 3 * nk + L + 2 * nl + nr + (sweep ? nk + nl : 0);
    HIPCHK(hipMalloc(&c->d_chain, total * sizeof(int32_t)));
    int32_t *p = static_cast<int32_t *>(c->d_chain);
    size_t off = 0;
    auto put = [&](const std::vector<int32_t> &v) -> const int32_t * {
        int32_t *dst = p + off;
        off += v.size();
        return hipMemcpy(dst, v.data(), v.size() * sizeof(int32_t), hipMemcpyHostToDevice) == hipSuccess
                   ? dst
                   : nullptr;
    };
    c->dc.L = L;
    c->dc.K = K;
    c->dc.x = put(c->h.x);
    c->dc.xbar = put(c->run.xbar);
    c->dc.c1 = put(c->run.c1);
    c->dc.need1 = put(c->run.need1);
    c->dc.need1max = put(c->run.need1max);
    c->dc.P = put(c->h.P);
    c->dc.need2 = put(c->h.need2);
    c->dc.lb = put(c->h.lb);
    c->dc.c3 = sweep ? put(c->run.c3) : nullptr;
    c->dc.need3 = sweep ? put(c->h.need3) : nullptr;
    c->dc.h_msa = c->h.msa.data();
    c->dc.h_msaH = sweep ? c->h.msaH.data() : nullptr;
    int64_t xbar_max = 0;
    for (int32_t v : c->run.xbar) xbar_max = std::max<int64_t>(xbar_max, v);
    c->dc.xbar_halo = xbar_max > rk::HMAX ? rk::HMAX + 1 : rk::round64(xbar_max);
    if (!c->dc.x || !c->dc.xbar || !c->dc.c1 || !c->dc.need1 || !c->dc.need1max || !c->dc.P ||
        !c->dc.need2 || !c->dc.lb || (sweep && (!c->dc.c3 || !c->dc.need3))) {  // leave no half-uploaded arrays behind: the next solve uploads again
        (void)hipFree(c->d_chain);
        c->d_chain = nullptr;
        return RK_E_DEVICE;
    }
    // each created once; a call that failed half way creates the rest next time
    if (!c->ev_fill0) HIPCHK(hipEventCreate(&c->ev_fill0));
    if (!c->ev_fill1) HIPCHK(hipEventCreate(&c->ev_fill1));
    if (!c->own_stream) HIPCHK(hipStreamCreateWithFlags(&c->own_stream, hipStreamNonBlocking));
    if (!c->d_res && hipMalloc(&c->d_res, 4 * sizeof(int64_t)) != hipSuccess) {
        c->d_res = nullptr;
        return RK_E_NOMEM;
    }
    return RK_OK;
}

int32_t to_abi(int32_t v) { return v >= DINF ? RK_INF : v; }

// Tables of rk_solve_noalloc: a static array on every device the library runs on.  In host
// code its name stands for a host-side shadow, not for device memory: the device address
// comes from hipGetSymbolAddress, once per device, with that device current, and only
// that address is handed to kernels.
static __device__ __align__(256) int32_t scratch[RK_NOALLOC_MAX_BYTES / sizeof(int32_t)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device `dev`.
int scratch_address(int dev, void **ptr)
{
    if (dev < 0 || dev >= kMaxDevices) return RK_E_DEVICE;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return RK_E_DEVICE;
        }
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return RK_OK;
}

// Queue the fill on `stream`: replay the captured launch sequence when nothing it depends
// on changed, else capture it anew.  With `direct` the kernels are launched one by one
// (inside a capture of the caller's they go into that capture; rk_solve_noalloc may not
// create a graph).
int fill(rk_chain *c, int32_t M, const Geometry &g, int32_t *tables, hipStream_t stream, bool direct = false)
{
    c->queued = false;
    c->M = M;
    c->W = g.W;
    c->tb.W = g.W;
    c->tb.padl = g.padl;
    c->tb.stride = g.stride;
    c->tb.inf_row = g.rows - 1;
    const int64_t tsz = rk::table_rows(c->h.L) * (int64_t)g.stride;
    c->tb.opt = tables + rk::SLACK * (int64_t)g.stride;
    c->tb.ap = c->tb.opt + tsz;
    c->tb.os = c->tb.ap + tsz;
    c->tb.hopt = c->dc.c3 ? c->tb.os + tsz : nullptr;
    c->tb.aq = c->dc.c3 ? c->tb.os + 2 * tsz : nullptr;
    // profiled fills launch their kernels one by one, never inside a graph: with counting on,
    // the counting variants of the kernels add what only they know (evaluated and skipped
    // candidates) into a small device array
    if (c->prof.count && !c->prof.d_ctr)
        HIPCHK(hipMalloc(&c->prof.d_ctr, rk::CTR_WORDS * sizeof(unsigned long long)));
    c->tb.ctr = c->prof.count ? c->prof.d_ctr : nullptr;
    c->tb.rec = nullptr;  // the fill points it at the profiler's records per launch (mode 2)
    c->prof.ctr_valid = c->prof.count;
    c->stream = stream;
    hipStreamCaptureStatus scs = hipStreamCaptureStatusNone;
    HIPCHK(hipStreamIsCapturing(stream, &scs));
    c->in_caller_graph = scs != hipStreamCaptureStatusNone;
    if (!c->in_caller_graph) HIPCHK(hipEventRecord(c->ev_fill0, stream));
    const bool replay = c->gexec && c->g_M == M && c->g_tables == tables && c->g_stream == stream &&
                        c->g_prof == c->prof.on;
    if (direct) {
        c->prof.reset(stream);
        HIPCHK(rk::launch_fill(c->dc, c->tb, stream, &c->launches, &c->prof));
    } else if (replay) {
        HIPCHK(hipGraphLaunch(c->gexec, stream));
    } else {
        if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
        c->gexec = nullptr;
        c->prof.reset(stream);
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        bool captured = false;
        // per-launch profiling events must be recorded on the stream itself (elapsed times
        // of events recorded inside a graph are not available), so profiled fills launch
        // directly
        if (!c->prof.on && hipStreamIsCapturing(stream, &cs) == hipSuccess &&
            cs == hipStreamCaptureStatusNone &&
            hipStreamBeginCapture(stream, hipStreamCaptureModeThreadLocal) == hipSuccess) {
            const hipError_t le = rk::launch_fill(c->dc, c->tb, stream, &c->launches, &c->prof);
            hipGraph_t graph = nullptr;
            const hipError_t ce = hipStreamEndCapture(stream, &graph);
            if (le == hipSuccess && ce == hipSuccess && graph &&
                hipGraphInstantiate(&c->gexec, graph, nullptr, nullptr, 0) == hipSuccess) {
                captured = true;
                c->g_M = M;
                c->g_tables = tables;
                c->g_stream = stream;
                c->g_prof = c->prof.on;
            }
            if (graph) (void)hipGraphDestroy(graph);
            (void)hipGetLastError();
        }
        if (captured) {
            HIPCHK(hipGraphLaunch(c->gexec, stream));
        } else {  // the stream is being captured by the caller, or capture is unavailable
            c->gexec = nullptr;
            c->prof.reset(stream);
            HIPCHK(rk::launch_fill(c->dc, c->tb, stream, &c->launches, &c->prof));
        }
    }
    if (!c->in_caller_graph) HIPCHK(hipEventRecord(c->ev_fill1, stream));
    c->queued = true;
    ++c->fills;
    return RK_OK;
}

int answer(rk_chain *c, int32_t *out)
{
    if (!c->queued) return RK_E_NOT_SOLVED;
    HIPCHK(wait_fill(c));
    if (c->M < c->h.x[0]) { *out = RK_INF; return RK_OK; }
    int32_t v = 0;
    const int64_t idx = rk::row_of(c->h.L, 0, c->h.L - 1) * c->tb.stride + c->tb.padl + (c->M - c->h.x[0]);
    HIPCHK(hipMemcpy(&v, c->tb.opt + idx, sizeof(int32_t), hipMemcpyDeviceToHost));
    *out = to_abi(v);
    return RK_OK;
}

}  // namespace

extern "C" {

int rk_chain_create(int32_t L, int32_t K, const int32_t *x, const int32_t *fn_time,
                    const int32_t *fn_tmp, const int32_t *fwd, const int32_t *bwd,
                    const int32_t *mem, const int32_t *tmp_fwd, const int32_t *tmp_bwd,
                    rk_chain **out)
{
    if (!out) return RK_E_INVAL;
    *out = nullptr;
    rk_chain *c = new (std::nothrow) rk_chain;
    if (!c) return RK_E_NOMEM;
    int rc;
    try {
        rc = rk::host_create(c->h, L, K, x, fn_time, fn_tmp, fwd, bwd, mem, tmp_fwd, tmp_bwd);
    } catch (...) {
        rc = RK_E_NOMEM;
    }
    if (rc != RK_OK) {
        delete c;
        return rc;
    }
    *out = c;
    return RK_OK;
}

int rk_chain_set_saving_sweep(rk_chain *c, const int32_t *refwd)
{
    if (!c) return RK_E_INVAL;
    int rc;
    try {
        rk::HostChain h = c->h;  // left unchanged on an error
        rc = rk::host_set_refwd(h, refwd);
        if (rc == RK_OK) {
            c->h.refwd.swap(h.refwd);
            c->h.c3.swap(h.c3);
            c->h.need3.swap(h.need3);
            c->h.msaH.swap(h.msaH);
            c->h.kept.swap(h.kept);
        }
    } catch (...) {
        rc = RK_E_NOMEM;
    }
    if (rc == RK_OK) ++c->host_version;  // the next solve rebuilds the device arrays
    return rc;
}

void rk_chain_destroy(rk_chain *c)
{
    if (!c) return;
    if (c->device >= 0) {  // something may live on the chain's device
        DeviceScope ds(c);
        if (c->queued && c->ev_fill1) (void)wait_fill(c);
        if (c->d_chain) (void)hipFree(c->d_chain);
        if (c->own_ws) (void)hipFree(c->own_ws);
        if (c->d_ops) (void)hipFree(c->d_ops);
        if (c->d_res) (void)hipFree(c->d_res);
        if (c->d_argrow) (void)hipFree(c->d_argrow);
        if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
        if (c->ev_fill0) (void)hipEventDestroy(c->ev_fill0);
        if (c->ev_fill1) (void)hipEventDestroy(c->ev_fill1);
        if (c->own_stream) (void)hipStreamDestroy(c->own_stream);
        for (hipEvent_t e : c->prof.events) (void)hipEventDestroy(e);
        if (c->prof.d_ctr) (void)hipFree(c->prof.d_ctr);
        if (c->prof.d_rec) (void)hipFree(c->prof.d_rec);
    }
    delete c;
}

int rk_workspace_bytes(const rk_chain *c, int32_t M, size_t *bytes)
{
    if (!c || !bytes) return RK_E_INVAL;
    Geometry g;
    return geometry(c, M, &g, bytes);
}

int rk_solve_async(rk_chain *c, int32_t M, void *d_workspace, size_t ws_bytes, void *stream)
{
    if (!c) return RK_E_INVAL;
    size_t need = 0;
    Geometry g;
    int rc = geometry(c, M, &g, &need);
    if (rc != RK_OK) return rc;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    // Inside a capture of the caller's stream nothing may allocate, upload or wait: the
    // chain must be set up by an earlier solve, and the tables are the caller's.
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (stream && hipStreamIsCapturing(static_cast<hipStream_t>(stream), &cs) != hipSuccess) return RK_E_DEVICE;
    if (cs != hipStreamCaptureStatusNone) {
        if (!c->d_chain || c->run_prune != c->prune || c->run_version != c->host_version || !d_workspace ||
            c->prof.on)
            return RK_E_INVAL;
        if (ws_bytes < need) return RK_E_NOMEM;
        return fill(c, M, g, static_cast<int32_t *>(d_workspace), static_cast<hipStream_t>(stream), true);
    }
    if ((rc = ensure_device(c)) != RK_OK) return rc;
    if (c->queued) HIPCHK(wait_fill(c));  // previous fill may still read its table
    int32_t *tab;
    if (d_workspace) {
        if (ws_bytes < need) return RK_E_NOMEM;
        tab = static_cast<int32_t *>(d_workspace);
    } else {
        if (c->own_ws_bytes < need) {
            if (c->own_ws) HIPCHK(hipFree(c->own_ws));
            c->own_ws = nullptr;
            c->own_ws_bytes = 0;
            if (hipMalloc(&c->own_ws, need) != hipSuccess) {
                (void)hipGetLastError();
                c->queued = false;
                return RK_E_NOMEM;
            }
            c->own_ws_bytes = need;
        }
        tab = static_cast<int32_t *>(c->own_ws);
    }
    return fill(c, M, g, tab, stream ? static_cast<hipStream_t>(stream) : c->own_stream);
}

int rk_solve_noalloc(rk_chain *c, int32_t M, void *stream)
{
    if (!c) return RK_E_INVAL;
    size_t need = 0;
    Geometry g;
    int rc = geometry(c, M, &g, &need);
    if (rc != RK_OK) return rc;
    if (need > RK_NOALLOC_MAX_BYTES) return RK_E_NOMEM;
    // the derived arrays, events and stream exist from an earlier solve on this device
    if (!c->d_chain || c->run_prune != c->prune || c->run_version != c->host_version || c->prof.on ||
        !c->ev_fill0 || !c->ev_fill1)
        return RK_E_INVAL;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    void *tab = nullptr;
    if ((rc = scratch_address(c->device, &tab)) != RK_OK) return rc;
    if (c->queued) HIPCHK(wait_fill(c));  // the previous fill may still read its table
    // launched directly: capturing and instantiating a graph would allocate
    return fill(c, M, g, static_cast<int32_t *>(tab), stream ? static_cast<hipStream_t>(stream) : c->own_stream,
                true);
}

int rk_solve(rk_chain *c, int32_t M, int32_t *opt_out)
{
    if (!c || !opt_out) return RK_E_INVAL;
    int rc = rk_solve_async(c, M, nullptr, 0, nullptr);
    if (rc != RK_OK) return rc;
    DeviceScope ds(c);
    return answer(c, opt_out);
}

int rk_result(rk_chain *c, int32_t *opt_out)
{
    if (!c || !opt_out) return RK_E_INVAL;
    if (!c->queued) return RK_E_NOT_SOLVED;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    return answer(c, opt_out);
}

int rk_extract_schedule(rk_chain *c, rk_op *ops, int64_t cap, int64_t *n_ops, int64_t *n_fwd)
{
    if (!c || !n_ops || cap < 0) return RK_E_INVAL;
    if (!c->queued) return RK_E_NOT_SOLVED;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    int32_t ans = 0;
    int rc = answer(c, &ans);
    if (rc != RK_OK) return rc;
    if (ans == RK_INF) return RK_E_INFEASIBLE;
    // At most L forwards per block (one saving) and one backward, one forget per no-save forward.
    // At most L forwards per block (one saving, one re-forward with the saving sweep) and one
    // backward, one forget per no-save forward.
    const int64_t max_ops = 3 * (int64_t)c->h.L * c->h.L + 16;
    if (c->d_ops_cap < max_ops) {
        if (c->d_ops) HIPCHK(hipFree(c->d_ops));
        c->d_ops = nullptr;
        c->d_ops_cap = 0;
        c->bt_fill = -1;
        if (hipMalloc(&c->d_ops, max_ops * sizeof(rk_op)) != hipSuccess) return RK_E_NOMEM;
        c->d_ops_cap = max_ops;
    }
    // the schedule of this solve is computed once (the two-call protocol asks twice)
    int64_t *const res = c->bt_res;
    if (c->bt_fill != c->fills) {
        c->bt_fill = -1;
        HIPCHK(rk::launch_backtrace(c->dc, c->tb, c->M - c->h.x[0], c->d_ops, c->d_ops_cap, c->d_res,
                                    c->stream));
        HIPCHK(hipMemcpyAsync(res, c->d_res, 3 * sizeof(int64_t), hipMemcpyDeviceToHost, c->stream));
        HIPCHK(hipStreamSynchronize(c->stream));
        c->bt_fill = c->fills;
    }
    if (res[2] != 0 || res[0] > c->d_ops_cap) return RK_E_INTERNAL;
    *n_ops = res[0];
    if (n_fwd) *n_fwd = res[1];
    if (!ops || cap < res[0]) return RK_E_BUFSZ;
    HIPCHK(hipMemcpy(ops, c->d_ops, res[0] * sizeof(rk_op), hipMemcpyDeviceToHost));
    for (int64_t k = 0; k < res[0]; ++k)  // option slots back to the caller's option indices
        if (ops[k].kind == RK_FWD_SAVE || ops[k].kind == RK_BWD || ops[k].kind == RK_REFWD)
            ops[k].option = c->run.opt[(size_t)ops[k].block * c->run.k_run + ops[k].option];
    return RK_OK;
}

int rk_read_row(rk_chain *c, int32_t s, int32_t t, int32_t *opt_row, int16_t *arg_row)
{
    if (!c || s < 0 || t < s || t >= c->h.L) return RK_E_INVAL;
    if (!c->queued) return RK_E_NOT_SOLVED;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    HIPCHK(wait_fill(c));
    const int64_t base = rk::row_of(c->h.L, s, t) * c->tb.stride + c->tb.padl;
    if (opt_row) {
        HIPCHK(hipMemcpy(opt_row, c->tb.opt + base, (size_t)c->W * sizeof(int32_t), hipMemcpyDeviceToHost));
        for (int32_t m = 0; m < c->W; ++m) opt_row[m] = to_abi(opt_row[m]);
    }
    if (arg_row) {
        if (c->d_argrow_cap < c->W) {
            if (c->d_argrow) HIPCHK(hipFree(c->d_argrow));
            c->d_argrow = nullptr;
            c->d_argrow_cap = 0;
            if (hipMalloc(&c->d_argrow, (size_t)c->W * sizeof(int16_t)) != hipSuccess) return RK_E_NOMEM;
            c->d_argrow_cap = c->W;
        }
        HIPCHK(rk::launch_arg_row(c->dc, c->tb, s, t, c->d_argrow, c->stream));
        HIPCHK(hipMemcpyAsync(arg_row, c->d_argrow, (size_t)c->W * sizeof(int16_t),
                              hipMemcpyDeviceToHost, c->stream));
        HIPCHK(hipStreamSynchronize(c->stream));
        for (int32_t m = 0; m < c->W; ++m)  // option slots back to the caller's option indices
            if (arg_row[m] >= c->h.L + c->run.k_run)  // case 3 (the saving sweep)
                arg_row[m] = (int16_t)(c->h.L + c->h.K +
                                       c->run.opt[(size_t)s * c->run.k_run + (arg_row[m] - c->h.L - c->run.k_run)]);
            else if (arg_row[m] >= c->h.L)
                arg_row[m] = (int16_t)(c->h.L + c->run.opt[(size_t)s * c->run.k_run + (arg_row[m] - c->h.L)]);
    }
    return RK_OK;
}

int rk_tradeoff_curve(rk_chain *c, int32_t *times, int64_t n)
{
    if (!c || (!times && n > 0) || n < 0) return RK_E_INVAL;
    if (!c->queued) return RK_E_NOT_SOLVED;
    if (n > (int64_t)c->W) return RK_E_INVAL;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    HIPCHK(wait_fill(c));
    // budget b leaves b - x_0 slots beyond the chain input: Opt(0, L-1, b - x_0)
    const int64_t x0 = c->h.x[0], lead = std::min<int64_t>(n, x0);
    for (int64_t b = 0; b < lead; ++b) times[b] = RK_INF;
    if (n > x0) {
        const int64_t base = rk::row_of(c->h.L, 0, c->h.L - 1) * c->tb.stride + c->tb.padl;
        HIPCHK(hipMemcpy(times + x0, c->tb.opt + base, (size_t)(n - x0) * sizeof(int32_t), hipMemcpyDeviceToHost));
        for (int64_t b = x0; b < n; ++b) times[b] = to_abi(times[b]);
    }
    return RK_OK;
}

int rk_last_fill_ms(rk_chain *c, float *ms, int32_t *launches)
{
    if (!c || !ms) return RK_E_INVAL;
    if (!c->queued) return RK_E_NOT_SOLVED;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    if (c->in_caller_graph) return RK_E_INVAL;
    HIPCHK(hipEventSynchronize(c->ev_fill1));
    HIPCHK(hipEventElapsedTime(ms, c->ev_fill0, c->ev_fill1));
    if (launches) *launches = c->launches;
    return RK_OK;
}

int rk_set_profiling(rk_chain *c, int32_t mode)
{
    if (!c || mode < 0 || mode > 2) return RK_E_INVAL;
    c->prof.on = mode != 0;
    c->prof.count = mode == 2;
    return RK_OK;
}

int rk_fill_kernel_stats(rk_chain *c, int32_t kind, int32_t *n_kinds, const char **name,
                         int32_t *launches, float *total_ms, int64_t *relaxations, int64_t *evaluated,
                         int64_t *bytes)
{
    if (!c) return RK_E_INVAL;
    if (n_kinds) *n_kinds = rk::KFILL_NKINDS;
    if (kind < 0 || kind >= rk::KFILL_NKINDS) return RK_E_INVAL;
    if (name) *name = rk::kFillKernelNames[kind];
    if (!c->queued) return RK_E_NOT_SOLVED;
    DeviceScope ds(c);
    if (!ds.ok) return RK_E_DEVICE;
    HIPCHK(wait_fill(c));
    int32_t cnt = 0;
    float sum = 0.f;
    for (int32_t j = 0; j < c->prof.n; ++j) {
        if (c->prof.kinds[j] != kind) continue;
        float ms = 0.f;
        HIPCHK(hipEventElapsedTime(&ms, c->prof.events[2 * j], c->prof.events[2 * j + 1]));
        sum += ms;
        ++cnt;
    }
    if (launches) *launches = cnt;
    if (total_ms) *total_ms = sum;
    if (relaxations) *relaxations = c->prof.work[kind];
    // the finalize's skips (mode 2): candidates of near splits that the lower bound
    // lb(s,t) + P(s,i) let a wave skip, each sparing two 4-byte operand reads
    int64_t skipped = 0;
    if (kind == rk::KFILL_FINALIZE && c->prof.ctr_valid && c->prof.d_ctr && (evaluated || bytes)) {
        std::vector<unsigned long long> ctr(rk::CTR_WORDS);
        HIPCHK(hipMemcpy(ctr.data(), c->prof.d_ctr, ctr.size() * sizeof ctr[0], hipMemcpyDeviceToHost));
        for (int32_t j = 0; j < rk::CTR_SLOTS; ++j) skipped += (int64_t)ctr[(int64_t)j * rk::CTR_PITCH];
    }
    if (evaluated) *evaluated = c->prof.eval[kind] - skipped;
    if (bytes) *bytes = c->prof.bytes[kind] - 8 * skipped;
    return RK_OK;
}

int rk_set_option_pruning(rk_chain *c, int32_t enable)
{
    if (!c) return RK_E_INVAL;
    c->prune = enable != 0;
    return RK_OK;
}

int rk_chain_options(const rk_chain *c, int32_t *kept, int32_t *k_run)
{
    if (!c) return RK_E_INVAL;
    int32_t kr = 1;
    for (int32_t s = 0; s < c->h.L; ++s) {
        int32_t n = 0;
        for (int32_t o = 0; o < c->h.K; ++o) {
            const size_t j = (size_t)s * c->h.K + o;
            const int32_t v = !c->prune || c->h.kept[j];
            if (kept) kept[j] = v;
            n += v;
        }
        kr = std::max(kr, n);
    }
    if (k_run) *k_run = kr;
    return RK_OK;
}

const char *rk_strerror(int code)
{
    switch (code) {
    case RK_OK: return "ok";
    case RK_E_INVAL: return "invalid argument";
    case RK_E_OVERFLOW: return "schedule times could exceed RK_TIME_LIMIT";
    case RK_E_NOMEM: return "allocation failed or workspace too small";
    case RK_E_DEVICE: return "HIP device error";
    case RK_E_NOT_SOLVED: return "no solve to read from";
    case RK_E_INFEASIBLE: return "budget admits no schedule";
    case RK_E_BUFSZ: return "buffer too small";
    case RK_E_INTERNAL: return "internal consistency check failed";
    default: return "unknown error";
    }
}

}  // extern "C"
