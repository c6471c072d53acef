// C-ABI entry points of the block-quantized linear library (include/qlinear.h):
// argument checks, tile-shape choice and launch.  Every check happens before
// anything is enqueued; no entry point throws or aborts.
#include <algorithm>
#include <atomic>
#include <functional>
#include <mutex>
#include <queue>
#include <vector>

#include "epilogue.h"
#include "internal.h"

using namespace qlk;

namespace {

constexpr int64_t I31 = (int64_t)1 << 31;

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool fmt_ok(int f) { return f == QL_FMT_INT8 || f == QL_FMT_Q4; }

// formats the forward product takes: the quantized ones and fp16 weights
bool fwd_fmt_ok(int f) { return fmt_ok(f) || f == QL_FMT_F16; }

int check_linear(int fmt, const void *X, int xdt, int64_t M, int64_t K, const void *codes,
                 const uint16_t *scales, int64_t N, const void *Y, int ydt = QL_DT_F32)
{
    const bool f16 = fmt == QL_FMT_F16;
    if (!fwd_fmt_ok(fmt) || (xdt != QL_DT_F32 && xdt != QL_DT_BF16))
        return QL_ERR_INVALID;
    if (M < 0 || N <= 0 || K <= 0 || K % QL_BLOCK)
        return QL_ERR_SHAPE;
    if (M >= I31 || N >= I31 || K >= I31)
        return QL_ERR_UNSUPPORTED;
    // fp16 weights: the fp16 path's kernel only (bf16 X, whole 256-k steps)
    if (f16 && (xdt != QL_DT_BF16 || K % 256 || K >= ((int64_t)1 << 22)))
        return QL_ERR_UNSUPPORTED;
    if (!codes || (!f16 && !scales) || (M > 0 && (!X || !Y)))
        return QL_ERR_INVALID;
    if (!aligned(codes, 16) || (!f16 && !aligned(scales, 2)) ||
        (M > 0 && (!aligned(X, 16) || !aligned(Y, ydt == QL_DT_BF16 ? 2 : 4))))
        return QL_ERR_ALIGN;
    return QL_OK;
}

const ql_epilogue NO_EPILOGUE = {nullptr, QL_ACT_NONE, nullptr, QL_DT_F32, nullptr, 0.0f, nullptr,
                                 nullptr};

// an epilogue's enums, aliasing and alignment (before check_linear, which
// takes its ydt)
int check_epilogue(const ql_epilogue &ep, const void *Y)
{
    if ((ep.act != QL_ACT_NONE && ep.act != QL_ACT_GELU) ||
        (ep.ydt != QL_DT_F32 && ep.ydt != QL_DT_BF16))
        return QL_ERR_INVALID;
    // an in-place residual add needs fp32 Y
    if (ep.ydt == QL_DT_BF16 && ep.residual && (const void *)ep.residual == Y)
        return QL_ERR_INVALID;
    if (ep.steer_dir && !ep.steer_strength)
        return QL_ERR_INVALID;
    // the bf16 copy is of an fp32 output, and is an output of its own
    if (ep.y_bf16_copy && (ep.ydt != QL_DT_F32 || (const void *)ep.y_bf16_copy == Y ||
                           (const void *)ep.y_bf16_copy == ep.residual))
        return QL_ERR_INVALID;
    if (!aligned(ep.bias, 4) || !aligned(ep.residual, 4) || !aligned(ep.y_bf16_copy, 2) ||
        (ep.steer_dir && (!aligned(ep.steer_dir, 4) || !aligned(ep.steer_strength, 4))))
        return QL_ERR_ALIGN;
    return QL_OK;
}

int check_layer(const ql_linear_ep &l)
{
    const int st = check_epilogue(l.ep, l.lin.Y);
    if (st != QL_OK)
        return st;
    return check_linear(l.lin.fmt, l.lin.X, l.lin.xdt, l.lin.M, l.lin.K, l.lin.codes,
                        l.lin.scales, l.lin.N, l.lin.Y, l.ep.ydt);
}

Epilogue to_epilogue(const ql_epilogue &e)
{
    return Epilogue{e.bias,
                    e.residual,
                    e.steer_dir,
                    e.steer_dir ? e.steer_strength : nullptr,
                    e.steer_norm,
                    e.act,
                    e.ydt == QL_DT_BF16 ? 1 : 0,
                    e.y_bf16_copy};
}

// Stream-ordered pool (one per device) that the per-stream workspaces below
// come from.  The pool keeps what it has grown to.
hipMemPool_t workspace_pool()
{
    constexpr int MAXDEV = 64;
    static std::mutex mu;
    static hipMemPool_t pools[MAXDEV] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV)
        return nullptr;
    std::lock_guard<std::mutex> g(mu);
    if (!pools[dev]) {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t p = nullptr;
        if (hipMemPoolCreate(&p, &props) != hipSuccess)
            return nullptr;
        uint64_t keep = UINT64_MAX;
        if (hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep) != hipSuccess) {
            (void)hipMemPoolDestroy(p);  // already failing; nothing to report
            return nullptr;
        }
        pools[dev] = p;
    }
    return pools[dev];
}

size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

// Workspace of the large-M bf16 path (fp16 activation copies, split
// partials).  Calls on one stream run in order, so one buffer per (device,
// stream) serves them all; taking it costs nothing on the device, where a
// stream-ordered allocation and free per call cost microseconds (and, in a
// captured graph, allocation nodes that cost more).  The buffer grows, in
// stream order, when a call outside graph capture needs more; the old one is
// returned to the pool unless a graph was captured with it, in which case it
// stays allocated for the life of the process (replays still use it).  A
// call under capture that needs more than the stream's buffer takes a
// stream-ordered allocation for itself (freed after its launch) instead.
struct Workspace {
    uint8_t *ptr;
    bool own_alloc;  // allocated for this call: free after the launch
};

bool take_workspace(size_t bytes, hipStream_t stream, Workspace &w)
{
    struct Entry {
        int dev;
        hipStream_t stream;
        void *ptr;
        size_t bytes;
        bool captured;  // a graph holds this buffer
    };
    static std::mutex mu;
    static std::vector<Entry> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return false;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess)
        return false;
    const bool capturing = cs != hipStreamCaptureStatusNone;
    hipMemPool_t pool = workspace_pool();
    if (!pool)
        return false;
    std::lock_guard<std::mutex> g(mu);
    Entry *e = nullptr;
    for (Entry &c : cache)
        if (c.dev == dev && c.stream == stream)
            e = &c;
    if (!e) {
        cache.push_back(Entry{dev, stream, nullptr, 0, false});
        e = &cache.back();
    }
    if (e->bytes >= bytes) {
        e->captured |= capturing;
        w = Workspace{(uint8_t *)e->ptr, false};
        return true;
    }
    void *p = nullptr;
    if (capturing) {
        if (hipMallocFromPoolAsync(&p, bytes, pool, stream) != hipSuccess)
            return false;
        w = Workspace{(uint8_t *)p, true};
        return true;
    }
    const size_t grow = ((std::max(bytes, e->bytes + e->bytes / 2)) + ((size_t)1 << 21) - 1) &
                        ~(((size_t)1 << 21) - 1);
    if (hipMallocFromPoolAsync(&p, grow, pool, stream) != hipSuccess)
        return false;
    if (e->ptr && !e->captured && hipFreeAsync(e->ptr, stream) != hipSuccess) {
        (void)hipFreeAsync(p, stream);  // already failing; nothing to report
        return false;
    }
    *e = Entry{dev, stream, p, grow, false};
    w = Workspace{(uint8_t *)p, false};
    return true;
}

// Where a call's workspace comes from: the per-stream buffer above, or a
// fixed region (the no-allocation entry point's static scratch).  A dry run
// enqueues nothing: it only records the largest workspace the call takes.
struct WsSource {
    uint8_t *fixed;  // device address of the fixed region, or nullptr: pool
    size_t cap;      // bytes of the fixed region
    bool dry_run;
    size_t need;     // out: largest single request
};

WsSource pool_source() { return WsSource{nullptr, 0, false, 0}; }

bool get_workspace(WsSource &wsrc, size_t bytes, hipStream_t stream, Workspace &w)
{
    wsrc.need = std::max(wsrc.need, bytes);
    if (wsrc.fixed) {
        if (bytes > wsrc.cap)
            return false;
        w = Workspace{wsrc.fixed, false};
        return true;
    }
    return take_workspace(bytes, stream, w);
}

int device_cus()
{
    constexpr int MAXDEV = 64;
    static int cus[MAXDEV] = {};
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV)
        return 256;
    if (!cus[dev])
        cus[dev] = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) ==
                               hipSuccess && v > 0 ? v : 256;
    return cus[dev];
}

// Split plan of a grouped fp16-path launch: how many parts each layer's
// output tiles are cut into along K.  Tiles of different reduction lengths
// (FFN-down's K = 4d next to K = d) or too few tiles for the GPU leave most
// CUs idle at the end of the launch; cutting the long reductions into parts
// evens that out at the price of a partial-tile round trip per part.  The
// plan is the one with the shortest estimated makespan under the hardware's
// dispatch: workgroup p runs on XCD p % 8, each XCD takes a contiguous range
// of every layer's parts (in layer order) and starts them in order on its
// first free CU.  The model counts one slot per CU: two workgroups resident
// on one CU finish about as late as the two one after the other (measured
// on single layers at 2048 tokens: out projection in 2 parts, one per CU,
// 40 us, in 4 parts, two per CU, 49 us).  A layer with at least as many
// tiles as there are CUs is not cut (measured: QKV at 2048 tokens, 384
// tiles, 71 us whole and 91 us in 2 parts).
//
// A launch that fits in one wave of workgroup slots has no other work to
// hide the last parts' in-kernel reduction behind: there the parts may
// instead store plain partial outputs that one more launch adds up at
// full-chip bandwidth (ext), which also allows more and shorter parts.
struct SplitPlan {
    int S[QL_MAX_GROUP], psteps[QL_MAX_GROUP];
    bool ext;
};

constexpr int XCDS = 8;
constexpr double TILE_OVH = 3.0;   // prologue + epilogue, in 64-k steps
constexpr double SPLIT_OVH = 2.0;  // partial store / reload per part
// one-wave single-layer launches (times in steps of ~1 us, measured):
constexpr double PART_STORE = 2.5;       // a part's partial store and arrival
constexpr double TAIL_PER_PART = 2.2;    // last arriver's reload of one partial tile
constexpr double EXT_GAP = 2.0;          // the extra launch
constexpr double EXT_BYTES_PER_STEP = 5.0e6;  // bytes the sum launch moves per step
constexpr int EXT_MAX_SPLIT = 16;
// an in-kernel reduction whose layer has an epilogue: the last part to
// arrive also applies it (residual loads, bias, copies) while the rest of
// the GPU waits (measured: out projection with its residual add and bf16
// copy, 2 parts, 53 us reduced in the kernel, 48 us by the sum launch)
constexpr double EPI_TAIL = 12.0;

double makespan(const LinDesc *d, int n, const SplitPlan &pl, int slots)
{
    double worst = 0.0;
    for (int x = 0; x < XCDS; ++x) {
        // slot free times, earliest first
        std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
        for (int k = 0; k < slots; ++k)
            free_at.push(0.0);
        for (int i = 0; i < n; ++i) {
            const int64_t parts = (int64_t)d[i].tiles_m * d[i].tiles_n * pl.S[i];
            const int64_t q = parts / XCDS, r = parts % XCDS;
            const int64_t mine = q + (x < r ? 1 : 0);
            const double len = pl.psteps[i] + TILE_OVH + (pl.S[i] > 1 ? SPLIT_OVH : 0.0);
            for (int64_t t = 0; t < mine; ++t) {
                const double end = free_at.top() + len;
                free_at.pop();
                free_at.push(end);
                worst = std::max(worst, end);
            }
        }
    }
    return worst;
}

SplitPlan plan_splits(int fmt, const LinDesc *d, int n)
{
    (void)fmt;
    const int cus = device_cus();
    const int slots = std::max(1, cus / XCDS);
    SplitPlan best{};
    double best_t = 0.0;
    int best_parts = 0;
    // candidate part lengths: every layer's step count halved repeatedly
    std::vector<int> cand;
    for (int i = 0; i < n; ++i)
        for (int L = d[i].K / 64; L >= 8; L /= 2)
            cand.push_back(L);
    cand.push_back(1 << 30);  // no split
    for (const int L : cand) {
        SplitPlan pl{};
        int total_parts = 0;
        for (int i = 0; i < n; ++i) {
            const int ns = d[i].K / 64;
            // parts of a multiple of 4 steps (whole scale chunks), >= 8 steps;
            // a layer with a tile for every CU stays whole
            int ps = ns;
            if (L < ns && (int64_t)d[i].tiles_m * d[i].tiles_n < cus) {
                ps = std::max(8, (L + 3) & ~3);
                ps = std::min(ps, ns);
            }
            pl.psteps[i] = ps;
            pl.S[i] = (ns + ps - 1) / ps;
            if (pl.S[i] > wide_max_split()) {
                const int S = wide_max_split();
                pl.psteps[i] = ((ns + S - 1) / S + 3) & ~3;
                pl.S[i] = (ns + pl.psteps[i] - 1) / pl.psteps[i];
            }
            total_parts += pl.S[i];
        }
        const double t = makespan(d, n, pl, slots);
        if (best_parts == 0 || t < best_t * 0.98 ||
            (t <= best_t * 1.02 && total_parts < best_parts)) {
            best = pl;
            best_t = t;
            best_parts = total_parts;
        }
    }
    const int64_t wave = (int64_t)slots * XCDS;
    int64_t parts = 0;
    for (int i = 0; i < n; ++i)
        parts += (int64_t)d[i].tiles_m * d[i].tiles_n * best.S[i];
    if (parts > wave)
        return best;
    // one wave: the tail of the in-kernel reduction is the last arrivers'
    // reload of every partial tile, against plans whose parts a separate
    // launch adds up (every layer cut to one common part length)
    best_t = 0.0;
    for (int i = 0; i < n; ++i)
        best_t = std::max(best_t, best.psteps[i] + TILE_OVH +
                                      (best.S[i] > 1 ? PART_STORE + TAIL_PER_PART * best.S[i] +
                                                           (epi_active(d[i].ep) ? EPI_TAIL : 0.0)
                                                     : 0.0));
    std::vector<int> lens;
    for (int i = 0; i < n; ++i)
        for (int L = d[i].K / 64; L >= 4; L /= 2)
            lens.push_back(L);
    for (const int L : lens) {
        SplitPlan pl{};
        pl.ext = true;
        int64_t np = 0;
        int longest = 0, split = 0;
        double sum_bytes = 0.0;
        for (int i = 0; i < n; ++i) {
            const int ns = d[i].K / 64;
            int ps = (int64_t)d[i].tiles_m * d[i].tiles_n < cus
                         ? std::min(ns, std::max(4, (L + 3) & ~3)) : ns;
            int S = (ns + ps - 1) / ps;
            if (S > EXT_MAX_SPLIT) {
                ps = ((ns + EXT_MAX_SPLIT - 1) / EXT_MAX_SPLIT + 3) & ~3;
                S = (ns + ps - 1) / ps;
            }
            pl.S[i] = S;
            pl.psteps[i] = ps;
            np += (int64_t)d[i].tiles_m * d[i].tiles_n * S;
            longest = std::max(longest, ps);
            if (S > 1) {
                ++split;
                sum_bytes += (S + 1) * (double)d[i].M * d[i].N * 4;
            }
        }
        if (!split || np > wave)
            continue;
        const double t = longest + TILE_OVH + PART_STORE + EXT_GAP + sum_bytes / EXT_BYTES_PER_STEP;
        if (t < best_t * 0.95) {
            best = pl;
            best_t = t;
        }
    }
    return best;
}

// Recently used plans, keyed by the group's shapes (the search above costs
// tens of microseconds of host time).
SplitPlan cached_plan(int fmt, const LinDesc *d, int n)
{
    struct Entry {
        int n, cus, slots;
        int64_t shape[QL_MAX_GROUP][3];
        SplitPlan pl;
    };
    constexpr int SLOTS = 16;
    static std::mutex mu;
    static Entry cache[SLOTS];
    static int used = 0, next = 0;
    Entry key{};
    key.n = n;
    key.cus = device_cus();
    key.slots = wide_wgs_per_cu(fmt);
    for (int i = 0; i < n; ++i) {
        key.shape[i][0] = d[i].M;
        key.shape[i][1] = d[i].N;
        key.shape[i][2] = d[i].K;
    }
    {
        std::lock_guard<std::mutex> g(mu);
        for (int e = 0; e < used; ++e)
            if (cache[e].n == n && cache[e].cus == key.cus && cache[e].slots == key.slots &&
                std::equal(&cache[e].shape[0][0], &cache[e].shape[0][0] + 3 * n, &key.shape[0][0]))
                return cache[e].pl;
    }
    key.pl = plan_splits(fmt, d, n);
    std::lock_guard<std::mutex> g(mu);
    cache[next] = key;
    next = (next + 1) % SLOTS;
    used = std::min(used + 1, SLOTS);
    return key.pl;
}

TileCfg choose_tile(int64_t M, bool xf32)
{
    if (M <= 16)
        return TILE_M16;
    if (M <= 32)
        return TILE_M32;
    if (M <= 64 || xf32)
        return TILE_M64;
    return TILE_M128;
}

// Kernel path forced by qlinear_force_path (QL_PATH_AUTO: the dispatch
// below chooses).  Process-wide; read once per call.
std::atomic<int> g_forced_path{QL_PATH_AUTO};

// Few-row kernels, one launch per layer (bf16 activations, quantized
// weights).  Which kernel each layer takes, decided for every layer before
// anything is launched.
enum class RowPath { GEMV, STREAM, SKINNY };

bool stream_fits(const LinDesc &d)
{
    return d.M <= stream_max_m() && d.K % 256 == 0 && d.K <= stream_max_k() &&
           aligned(d.scales, 16);
}

// the large-M kernel's shape limits (bf16 X): whole 256-k steps, 16-byte
// scale chunks, 32-bit row offsets within a tile
bool wide_fits(const ql_linear &l)
{
    return l.xdt == QL_DT_BF16 && l.K % 256 == 0 && l.K < ((int64_t)1 << 23) &&
           (l.fmt == QL_FMT_F16 || aligned(l.scales, 16));
}

int launch_rows(const ql_linear_ep *const *ls, int n, int forced, WsSource &wsrc,
                hipStream_t stream)
{
    const int fmt = ls[0]->lin.fmt;
    LinDesc ds[QL_MAX_GROUP];
    RowPath path[QL_MAX_GROUP];
    for (int i = 0; i < n; ++i) {
        LinDesc &d = ds[i];
        d = LinDesc{};
        d.X = ls[i]->lin.X;
        d.codes = (const uint8_t *)ls[i]->lin.codes;
        d.scales = ls[i]->lin.scales;
        d.Y = ls[i]->lin.Y;
        d.ep = to_epilogue(ls[i]->ep);
        d.M = (int)ls[i]->lin.M;
        d.N = (int)ls[i]->lin.N;
        d.K = (int)ls[i]->lin.K;
        d.ksplit = 1;
        switch (forced) {
        case QL_PATH_GEMV:
            if (!gemv_ok(d))
                return QL_ERR_UNSUPPORTED;
            path[i] = RowPath::GEMV;
            break;
        case QL_PATH_STREAM:
            if (!stream_fits(d))
                return QL_ERR_UNSUPPORTED;
            path[i] = RowPath::STREAM;
            break;
        case QL_PATH_SKINNY:
            if (d.M > skinny_max_m())
                return QL_ERR_UNSUPPORTED;
            path[i] = RowPath::SKINNY;
            break;
        default:
            // the GEMV's time grows with the rows, the streaming kernel's
            // hardly below 8: at four rows of q4 the streaming kernel is ahead
            // (a d = 2048 block 17.1 against 19.7 us); int8, with twice the
            // code bytes per row, keeps the GEMV up to four rows (22.5 / 23.0)
            path[i] = gemv_ok(d) && !(fmt == QL_FMT_Q4 && d.M == 4 && stream_fits(d))
                          ? RowPath::GEMV
                          : stream_fits(d) ? RowPath::STREAM : RowPath::SKINNY;
        }
    }
    // the streaming layers: one launch over all of them, their K parts
    // planned together; the split layers' partials side by side in the
    // workspace, summed by one more launch
    LayerGroup sg{};
    StreamPlan sp{};
    size_t part_off[QL_MAX_GROUP], part_bytes = 0;
    for (int i = 0; i < n; ++i)
        if (path[i] == RowPath::STREAM)
            sg.d[sg.n++] = ds[i];
    if (sg.n > 0) {
        int S[QL_MAX_GROUP], P[QL_MAX_GROUP];
        sp = stream_plan(fmt, sg.d, sg.n, device_cus(), S, P);
        sg.begin[0] = 0;
        for (int j = 0; j < sg.n; ++j) {
            LinDesc &d = sg.d[j];
            d.ksplit = S[j];
            d.psteps = P[j];
            sg.begin[j + 1] = sg.begin[j] + (d.N + sp.rw - 1) / sp.rw * S[j];
            part_off[j] = part_bytes;
            if (S[j] > 1)
                part_bytes += round256((size_t)S[j] * d.M * d.N * 4);
        }
    }
    wsrc.need = std::max(wsrc.need, part_bytes);
    if (wsrc.dry_run || (wsrc.fixed && part_bytes > wsrc.cap))
        return wsrc.dry_run ? QL_OK : QL_ERR_UNSUPPORTED;

    // the GEMV layers: one launch per distinct row count
    bool done[QL_MAX_GROUP] = {};
    for (int i = 0; i < n; ++i) {
        if (path[i] != RowPath::GEMV || done[i])
            continue;
        LayerGroup g{};
        for (int j = i; j < n; ++j)
            if (path[j] == RowPath::GEMV && !done[j] && ds[j].M == ds[i].M) {
                g.d[g.n++] = ds[j];
                done[j] = true;
            }
        // longest rows first: their workgroups carry the most bytes, and
        // the short ones then fill the launch's tail
        std::stable_sort(g.d, g.d + g.n,
                         [](const LinDesc &x, const LinDesc &y) { return x.K > y.K; });
        if (launch_qgemv(fmt, g, stream) != hipSuccess)
            return QL_ERR_HIP;
    }
    if (sg.n > 0) {
        Workspace ws{};
        if (part_bytes > 0) {
            if (!get_workspace(wsrc, part_bytes, stream, ws))
                return QL_ERR_HIP;
            for (int j = 0; j < sg.n; ++j)
                if (sg.d[j].ksplit > 1)
                    sg.d[j].part = (float *)(ws.ptr + part_off[j]);
        }
        hipError_t e = launch_qgemm_stream(fmt, sp, sg, stream);
        if (e == hipSuccess && part_bytes > 0) {
            SplitSum sums[QL_MAX_GROUP];
            int ns = 0;
            for (int j = 0; j < sg.n; ++j)
                if (sg.d[j].ksplit > 1)
                    sums[ns++] = SplitSum{sg.d[j].part, sg.d[j].ksplit, sg.d[j].M, sg.d[j].N,
                                          sg.d[j].Y, sg.d[j].ep};
            e = launch_split_sum(sums, ns, stream);
        }
        if (ws.own_alloc) {
            const hipError_t ef = hipFreeAsync(ws.ptr, stream);
            e = e == hipSuccess ? ef : e;
        }
        if (e != hipSuccess)
            return QL_ERR_HIP;
    }
    for (int i = 0; i < n; ++i)
        if (path[i] == RowPath::SKINNY && launch_qgemm_skinny(fmt, ds[i], stream) != hipSuccess)
            return QL_ERR_HIP;
    return QL_OK;
}

// The tiled exact kernel over a group (LinDescs set up with ksplit = 1).
// A group with too few tiles for two workgroups per CU has its reductions
// cut into parts of one common length (at least 4 steps of 64 k), each
// layer into ceil(steps / length) parts; the parts' plain partial outputs
// are added, in part order, by the split-sum launch, which also applies
// the layers' epilogues.
int launch_tiled(int fmt, bool xf32, TileCfg t, GroupArgs &a, WsSource &wsrc,
                 hipStream_t stream)
{
    const int n = a.n;
    const int64_t target = 2 * (int64_t)device_cus();
    int64_t work = 0;
    for (int i = 0; i < n; ++i)
        work += (int64_t)a.d[i].tiles_m * a.d[i].tiles_n * ((a.d[i].K / 32 + 1) / 2);
    const int64_t L = std::max<int64_t>(4, (work + target - 1) / target);
    int64_t total = 0;
    size_t part_off[QL_MAX_GROUP], bytes = 0;
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        const int ns = (d.K / 32 + 1) / 2;  // 64-k steps, the last one possibly half
        int S = (int)std::min<int64_t>(EXT_MAX_SPLIT, (ns + L - 1) / L);
        d.psteps = (ns + S - 1) / S;
        d.ksplit = S = (ns + d.psteps - 1) / d.psteps;
        d.tile_begin = (int)total;
        total += (int64_t)d.tiles_m * d.tiles_n * S;
        part_off[i] = bytes;
        if (S > 1)
            bytes += round256((size_t)S * d.M * d.N * 4);
    }
    if (total >= I31)
        return QL_ERR_UNSUPPORTED;
    a.total_tiles = (int)total;
    wsrc.need = std::max(wsrc.need, bytes);
    if (wsrc.dry_run)
        return QL_OK;
    Workspace ws{};
    if (bytes > 0) {
        if (!get_workspace(wsrc, bytes, stream, ws))
            return wsrc.fixed ? QL_ERR_UNSUPPORTED : QL_ERR_HIP;
        for (int i = 0; i < n; ++i)
            if (a.d[i].ksplit > 1)
                a.d[i].part = (float *)(ws.ptr + part_off[i]);
    }
    hipError_t e = launch_qgemm(fmt, xf32, t, a, stream);
    if (e == hipSuccess && bytes > 0) {
        SplitSum sums[QL_MAX_GROUP];
        int ns = 0;
        for (int i = 0; i < n; ++i)
            if (a.d[i].ksplit > 1)
                sums[ns++] = SplitSum{a.d[i].part, a.d[i].ksplit, a.d[i].M, a.d[i].N, a.d[i].Y,
                                      a.d[i].ep};
        e = launch_split_sum(sums, ns, stream);
    }
    if (ws.own_alloc) {
        const hipError_t ef = hipFreeAsync(ws.ptr, stream);
        e = e == hipSuccess ? ef : e;
    }
    return e == hipSuccess ? QL_OK : QL_ERR_HIP;
}

// The mid-M kernel (qgemm_mid.hip: bf16 X, int8 / q4 weights, 128 x 128
// tiles) over a group of layers.  Plan: one common part length L (a
// multiple of 4 steps of 64 k) cuts each layer into ceil(steps / L) parts
// (at most MID_MAX_SPLIT); among the lengths from each layer's whole
// reduction halved down to 4 steps, the one with the smallest estimated
// time: the makespan of the parts on the resident workgroups (times in
// steps, a part costing its steps plus MID_OVH), plus, when a layer is
// split, the sum launch (MID_SUM_GAP and the bytes of the partials it reads
// and the outputs it writes).
constexpr double MID_OVH = 4.0;
constexpr double MID_SUM_GAP = 4.0;
constexpr double MID_SUM_BYTES_PER_STEP = 2.5e6;
constexpr int MID_MAX_SPLIT = 16;
// largest M the dispatch sends to the mid-M kernel (above it, the large-M
// kernel's wider tiles and fp16 fold win)
constexpr int64_t MID_MAX_M = 256;
// (measured crossover, q4 blocks at 214 rows: d = 1024 with 12 steps per CU
// is 1.12x faster here, d = 1536 with 27 is 1.2x slower)
constexpr double MID_MAX_STEPS_PER_CU = 16.0;

bool mid_fits(const ql_linear &l)
{
    return l.xdt == QL_DT_BF16 && (l.fmt == QL_FMT_INT8 || l.fmt == QL_FMT_Q4) &&
           l.K % 256 == 0 && l.K < ((int64_t)1 << 23) && aligned(l.X, 16) &&
           aligned(l.codes, 16) && aligned(l.scales, 16);
}

void plan_mid(GroupArgs &a)
{
    const int n = a.n;
    const int slots = mid_wgs_per_cu() * device_cus();
    std::vector<int> lens;
    for (int i = 0; i < n; ++i)
        for (int L = a.d[i].K / 64; L >= 4; L /= 2)
            lens.push_back(L & ~3);
    auto parts_of = [](const LinDesc &d, int L, int &S, int &ps) {
        const int ns = d.K / 64;
        S = std::min(MID_MAX_SPLIT, (ns + L - 1) / L);
        ps = ((ns + S - 1) / S + 3) & ~3;
        S = (ns + ps - 1) / ps;
    };
    double best_t = 0.0;
    int best_L = 0;
    for (const int L : lens) {
        if (L < 4)
            continue;
        // every XCD takes its share of each layer's parts (launch order:
        // longest reduction first); parts go to the earliest free slot
        double t = 0.0, sum_bytes = 0.0;
        bool split = false;
        for (int x = 0; x < XCDS; ++x) {
            std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
            for (int k = 0; k < slots / XCDS; ++k)
                free_at.push(0.0);
            for (int i = 0; i < n; ++i) {
                const LinDesc &d = a.d[i];
                int S, ps;
                parts_of(d, L, S, ps);
                if (x == 0 && S > 1) {
                    split = true;
                    sum_bytes += (S + 1) * (double)d.M * d.N * 4;
                }
                const int64_t parts = (int64_t)d.tiles_m * d.tiles_n * S;
                const int64_t mine = parts / XCDS + (x < parts % XCDS ? 1 : 0);
                for (int64_t q = 0; q < mine; ++q) {
                    const double e = free_at.top() + ps + MID_OVH;
                    free_at.pop();
                    free_at.push(e);
                    t = std::max(t, e);
                }
            }
        }
        if (split)
            t += MID_SUM_GAP + sum_bytes / MID_SUM_BYTES_PER_STEP;
        if (best_L == 0 || t < best_t) {
            best_t = t;
            best_L = L;
        }
    }
    for (int i = 0; i < n; ++i) {
        int S, ps;
        parts_of(a.d[i], best_L, S, ps);
        a.d[i].ksplit = S;
        a.d[i].psteps = ps;
    }
}

// ls: layers of one quantized format with bf16 X, mid_fits each.
int launch_mid(const ql_linear_ep *const *ls, int n, WsSource &wsrc, hipStream_t stream)
{
    const int bm = mid_tile_bm(), bn = mid_tile_bn();
    // longest reduction first, so the long tiles start early
    const ql_linear_ep *ord[QL_MAX_GROUP];
    std::copy(ls, ls + n, ord);
    std::stable_sort(ord, ord + n,
                     [](const ql_linear_ep *x, const ql_linear_ep *y) { return x->lin.K > y->lin.K; });
    GroupArgs a{};
    a.n = n;
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        d.X = ord[i]->lin.X;
        d.codes = (const uint8_t *)ord[i]->lin.codes;
        d.scales = ord[i]->lin.scales;
        d.Y = ord[i]->lin.Y;
        d.ep = to_epilogue(ord[i]->ep);
        d.M = (int)ord[i]->lin.M;
        d.N = (int)ord[i]->lin.N;
        d.K = (int)ord[i]->lin.K;
        d.tiles_m = (int)((ord[i]->lin.M + bm - 1) / bm);
        d.tiles_n = (int)((ord[i]->lin.N + bn - 1) / bn);
    }
    plan_mid(a);
    int64_t total = 0;
    size_t part_off[QL_MAX_GROUP], bytes = 0;
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        d.tile_begin = (int)total;
        total += (int64_t)d.tiles_m * d.tiles_n * d.ksplit;
        part_off[i] = bytes;
        if (d.ksplit > 1)
            bytes += round256((size_t)d.ksplit * d.M * d.N * 4);
    }
    if (total >= I31)
        return QL_ERR_UNSUPPORTED;
    a.total_tiles = (int)total;
    wsrc.need = std::max(wsrc.need, bytes);
    if (wsrc.dry_run)
        return QL_OK;
    Workspace ws{};
    if (bytes > 0) {
        if (!get_workspace(wsrc, bytes, stream, ws))
            return wsrc.fixed ? QL_ERR_UNSUPPORTED : QL_ERR_HIP;
        for (int i = 0; i < n; ++i)
            if (a.d[i].ksplit > 1)
                a.d[i].part = (float *)(ws.ptr + part_off[i]);
    }
    hipError_t e = launch_qgemm_mid(ord[0]->lin.fmt, a, stream);
    if (e == hipSuccess && bytes > 0) {
        SplitSum sums[QL_MAX_GROUP];
        int ns = 0;
        for (int i = 0; i < n; ++i)
            if (a.d[i].ksplit > 1)
                sums[ns++] = SplitSum{a.d[i].part, a.d[i].ksplit, a.d[i].M, a.d[i].N, a.d[i].Y,
                                      a.d[i].ep};
        e = launch_split_sum(sums, ns, stream);
    }
    if (ws.own_alloc) {
        const hipError_t ef = hipFreeAsync(ws.ptr, stream);
        e = e == hipSuccess ? ef : e;
    }
    return e == hipSuccess ? QL_OK : QL_ERR_HIP;
}

// One grouped launch over layers that share fmt and xdt (M > 0 each).
int launch_group(const ql_linear_ep *const *ls, int n, WsSource &wsrc, hipStream_t stream)
{
    if (n == 0)
        return QL_OK;
    const bool xf32 = ls[0]->lin.xdt == QL_DT_F32;
    int64_t maxM = 0;
    for (int i = 0; i < n; ++i)
        maxM = std::max(maxM, ls[i]->lin.M);
    const bool f16 = ls[0]->lin.fmt == QL_FMT_F16;
    // fp16 weights have one kernel; a forced path applies to quantized ones
    const int forced = f16 ? QL_PATH_AUTO : g_forced_path.load(std::memory_order_relaxed);
    // beyond the streaming kernel's rows the mid-M kernel takes every group
    // it fits: at 33-64 rows it is 2.5-3x faster than the per-layer exact
    // kernels (a d = 2048 block 37-43 us against 92-121)
    bool all_mid = true;
    for (int i = 0; i < n; ++i)
        all_mid = all_mid && mid_fits(ls[i]->lin);
    const bool per_layer = forced == QL_PATH_AUTO
                          ? !xf32 && !f16 &&
                                (maxM <= stream_max_m() || (maxM <= skinny_max_m() && !all_mid))
                          : forced == QL_PATH_GEMV || forced == QL_PATH_STREAM ||
                                forced == QL_PATH_SKINNY;
    if (per_layer && xf32)
        return QL_ERR_UNSUPPORTED;  // the few-row kernels take bf16 activations
    if (per_layer)
        return launch_rows(ls, n, forced, wsrc, stream);
    // a few hundred rows: the exact single-launch kernel where every layer
    // fits it and the group's work is short (its 64-k steps of 128 x 128
    // tiles, per CU, at most MID_MAX_STEPS_PER_CU; beyond that the large-M
    // path's wider tiles outweigh its pre-pass)
    if (forced == QL_PATH_MID || (forced == QL_PATH_AUTO && !xf32 && !f16 && maxM <= MID_MAX_M)) {
        bool ok = true, wide_ok = true;
        double steps = 0.0;
        for (int i = 0; i < n; ++i) {
            const ql_linear &l = ls[i]->lin;
            ok = ok && mid_fits(l);
            wide_ok = wide_ok && wide_fits(l);
            steps += (double)((l.M + mid_tile_bm() - 1) / mid_tile_bm()) *
                     ((l.N + mid_tile_bn() - 1) / mid_tile_bn()) * (l.K / 64);
        }
        // (at most 64 rows the alternative is not the large-M path but the
        // tiled exact kernel, slower at any length)
        if (forced == QL_PATH_AUTO && wide_ok && choose_tile(maxM, false) == TILE_M128 &&
            steps > MID_MAX_STEPS_PER_CU * device_cus())
            ok = false;
        if (ok)
            return launch_mid(ls, n, wsrc, stream);
        if (forced == QL_PATH_MID)
            return QL_ERR_UNSUPPORTED;
    }
    if (forced == QL_PATH_WIDE)
        for (int i = 0; i < n; ++i)
            if (!wide_fits(ls[i]->lin))
                return QL_ERR_UNSUPPORTED;
    maxM = 0;
    for (int i = 0; i < n; ++i)
        maxM = std::max(maxM, ls[i]->lin.M);
    const TileCfg t = choose_tile(maxM, xf32);
    // the fp16 path's kernel reads each weight row's scales as 16-byte
    // chunks and addresses a tile's rows with 32-bit offsets
    bool wide = !xf32 && t == TILE_M128;
    for (int i = 0; i < n; ++i)
        wide = wide && wide_fits(ls[i]->lin);
    if (forced == QL_PATH_WIDE || forced == QL_PATH_TILED)
        wide = forced == QL_PATH_WIDE;
    wide = wide || f16;  // fp16 weights: this kernel at every M (checked by check_linear)
    const int bm = wide ? wide_tile_bm() : tile_bm(t);
    const int bn = wide ? wide_tile_bn() : tile_bn(t);

    // longest reduction first, so the long tiles start early
    const ql_linear_ep *ord[QL_MAX_GROUP];
    std::copy(ls, ls + n, ord);
    std::stable_sort(ord, ord + n,
                     [](const ql_linear_ep *a, const ql_linear_ep *b) { return a->lin.K > b->lin.K; });

    GroupArgs a{};
    int64_t total = 0;
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        d.X = ord[i]->lin.X;
        d.codes = (const uint8_t *)ord[i]->lin.codes;
        d.scales = ord[i]->lin.scales;
        d.Y = ord[i]->lin.Y;
        d.ep = to_epilogue(ord[i]->ep);
        d.M = (int)ord[i]->lin.M;
        d.N = (int)ord[i]->lin.N;
        d.K = (int)ord[i]->lin.K;
        d.tiles_m = (int)((ord[i]->lin.M + bm - 1) / bm);
        d.tiles_n = (int)((ord[i]->lin.N + bn - 1) / bn);
        d.ksplit = 1;
        d.psteps = (int)(ord[i]->lin.K / 64);
    }
    SplitPlan pl{};
    if (wide)
        pl = cached_plan(ord[0]->lin.fmt, a.d, n);
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        if (wide) {
            d.ksplit = pl.S[i];
            d.psteps = pl.psteps[i];
        }
        d.tile_begin = (int)total;
        total += (int64_t)d.tiles_m * d.tiles_n * d.ksplit;
    }
    int64_t rows = 0;  // pre-pass grid bound (one workgroup per activation row)
    for (int i = 0; i < n; ++i)
        rows += a.d[i].M;
    if (total >= I31 || rows >= I31)
        return QL_ERR_UNSUPPORTED;
    a.n = n;
    a.total_tiles = (int)total;
    if (!wide)
        return launch_tiled(ord[0]->lin.fmt, xf32, t, a, wsrc, stream);

    // Workspace: one exact, row-shifted fp16 copy per distinct activation
    // tensor (layers reading the same X share it)
    int src[QL_MAX_GROUP];
    size_t xoff[QL_MAX_GROUP], bytes = 0;
    for (int i = 0; i < n; ++i) {
        src[i] = i;
        for (int j = 0; j < i; ++j)
            if (a.d[j].X == a.d[i].X && a.d[j].M == a.d[i].M && a.d[j].K == a.d[i].K) {
                src[i] = j;
                break;
            }
        if (src[i] == i) {
            xoff[i] = bytes;
            bytes += round256((size_t)a.d[i].M * a.d[i].K * 2) + round256((size_t)a.d[i].M * 4);
        }
    }
    // layers whose epilogue cannot take groups of four outputs write plain
    // fp32 partials, and the sum launch applies their epilogue
    bool any_part_out = false;
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        d.part_out = epi_active(d.ep) && !epi_vec_ok(d.ep, d.Y, d.N) ? 1 : 0;
        any_part_out = any_part_out || d.part_out;
    }
    // split layers: fp32 partials (tiles [tiles][S][BM * BN], or plain
    // outputs [S][M][N] for a plan summed by a separate launch), then the
    // arrival counters of the in-kernel reductions
    size_t poff[QL_MAX_GROUP], coff[QL_MAX_GROUP];
    int ncnt = 0;
    for (int i = 0; i < n; ++i) {
        const LinDesc &d = a.d[i];
        if (d.ksplit == 1 && !d.part_out)
            continue;
        poff[i] = bytes;
        bytes += round256(pl.ext || d.part_out
                              ? (size_t)d.ksplit * d.M * d.N * 4
                              : (size_t)d.tiles_m * d.tiles_n * d.ksplit * bm * bn * 4);
    }
    const size_t cnt_off = bytes;
    for (int i = 0; i < n; ++i) {
        if (a.d[i].ksplit == 1 || pl.ext || a.d[i].part_out)
            continue;
        coff[i] = cnt_off + (size_t)ncnt * 4;
        ncnt += a.d[i].tiles_m * a.d[i].tiles_n;
    }
    bytes += round256((size_t)ncnt * 4);
    // the weight-row shifts of int8 / q4 layers, [ksplit][tiles_n * bn] per
    // layer (set by the pre-pass; a tile's 256 shifts are one aligned KB)
    const bool quant = ord[0]->lin.fmt != QL_FMT_F16;
    size_t woff[QL_MAX_GROUP];
    for (int i = 0; i < n && quant; ++i) {
        woff[i] = bytes;
        bytes += round256((size_t)a.d[i].ksplit * a.d[i].tiles_n * bn * 4);
    }
    if (wsrc.dry_run) {
        wsrc.need = std::max(wsrc.need, bytes);
        return QL_OK;
    }
    Workspace ws{};
    if (!get_workspace(wsrc, bytes, stream, ws))
        return wsrc.fixed ? QL_ERR_UNSUPPORTED : QL_ERR_HIP;
    uint8_t *const wsb = ws.ptr;
    for (int i = 0; i < n; ++i)
        if (a.d[i].ksplit > 1 || a.d[i].part_out) {
            a.d[i].part = (float *)(wsb + poff[i]);
            a.d[i].cnt = pl.ext || a.d[i].part_out ? nullptr : (int *)(wsb + coff[i]);
        }
    // one pre-pass launch over every distinct activation tensor and the
    // weight-row shifts; it also clears the split counters
    XprepJob jobs[QL_MAX_GROUP];
    int njobs = 0;
    const void *xs[QL_MAX_GROUP];
    const int *es[QL_MAX_GROUP];
    for (int i = 0; i < n; ++i) {
        if (src[i] != i) {
            xs[i] = xs[src[i]];
            es[i] = es[src[i]];
            continue;
        }
        uint16_t *xh = (uint16_t *)(wsb + xoff[i]);
        int *ex = (int *)(wsb + xoff[i] + round256((size_t)a.d[i].M * a.d[i].K * 2));
        jobs[njobs++] = XprepJob{a.d[i].X, a.d[i].M, a.d[i].K, xh, ex};
        xs[i] = xh;
        es[i] = ex;
    }
    WshiftJob wjobs[QL_MAX_GROUP];
    int nw = 0;
    for (int i = 0; i < n; ++i) {
        LinDesc &d = a.d[i];
        d.wshift = nullptr;
        if (!quant)
            continue;
        d.wshift = (const int *)(wsb + woff[i]);
        d.wsld = d.tiles_n * bn;
        wjobs[nw++] = WshiftJob{d.scales, d.N, d.wsld, d.K / 32, d.ksplit, 2 * d.psteps,
                                ord[0]->lin.fmt == QL_FMT_INT8 ? 127 : 7, (int *)(wsb + woff[i])};
    }
    hipError_t e = launch_xprep(jobs, njobs, wjobs, nw, ord[0]->lin.fmt == QL_FMT_Q4,
                                (int *)(wsb + cnt_off), ncnt, stream);
    for (int i = 0; i < n; ++i) {
        a.d[i].X = xs[i];
        a.d[i].xexp = es[i];
    }
    if (e == hipSuccess)
        e = launch_qgemm_wide(ord[0]->lin.fmt, a, stream);
    if ((pl.ext || any_part_out) && e == hipSuccess) {
        SplitSum sums[QL_MAX_GROUP];
        int ns = 0;
        for (int i = 0; i < n; ++i)
            if ((pl.ext && a.d[i].ksplit > 1) || a.d[i].part_out)
                sums[ns++] = SplitSum{a.d[i].part, a.d[i].ksplit, a.d[i].M, a.d[i].N, a.d[i].Y,
                                      a.d[i].ep};
        e = launch_split_sum(sums, ns, stream);
    }
    const hipError_t ef = ws.own_alloc ? hipFreeAsync(ws.ptr, stream) : hipSuccess;
    return e == hipSuccess && ef == hipSuccess ? QL_OK : QL_ERR_HIP;
}

// The layers of a block call, partitioned by (fmt, xdt): each class is one
// launch_group call.
struct Classes {
    const ql_linear_ep *cls[6][QL_MAX_GROUP];
    int cnt[6];
};

int classify(const ql_linear_ep *lin, int n_lin, Classes &c)
{
    if (!lin || n_lin < 1 || n_lin > QL_MAX_GROUP)
        return QL_ERR_INVALID;
    for (int i = 0; i < n_lin; ++i) {
        const int st = check_layer(lin[i]);
        if (st != QL_OK)
            return st;
    }
    std::fill(c.cnt, c.cnt + 6, 0);
    for (int i = 0; i < n_lin; ++i) {
        const ql_linear &l = lin[i].lin;
        if (l.M == 0)
            continue;
        const int f = l.fmt == QL_FMT_Q4 ? 0 : l.fmt == QL_FMT_INT8 ? 1 : 2;
        const int k = 2 * f + (l.xdt == QL_DT_BF16 ? 1 : 0);
        c.cls[k][c.cnt[k]++] = &lin[i];
    }
    return QL_OK;
}

// Static scratch of the no-allocation entry point (the fp16 activation
// copies, row shifts, split partials and arrival counters that the pool
// workspace holds otherwise).  Each device the library runs on holds its own
// copy for the life of the process.  Host code must never use the array's
// name as an address: kernels and copies take the device address that
// hipGetSymbolAddress returns for the current device (scratch_base).
constexpr size_t SCRATCH_BYTES = (size_t)128 << 20;
static __device__ __align__(256) uint8_t scratch[SCRATCH_BYTES];

// Device address of this device's scratch, looked up once per device (with
// that device current); nullptr if the lookup fails.
uint8_t *scratch_base()
{
    constexpr int MAXDEV = 64;
    static std::mutex mu;
    static uint8_t *base[MAXDEV] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV)
        return nullptr;
    std::lock_guard<std::mutex> g(mu);
    if (!base[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
            return nullptr;
        base[dev] = (uint8_t *)p;
    }
    return base[dev];
}

}  // namespace

extern "C" {

size_t qlinear_codes_bytes(int fmt, int64_t N, int64_t K)
{
    if (!fwd_fmt_ok(fmt) || N <= 0 || K <= 0)
        return 0;
    return fmt == QL_FMT_INT8 ? (size_t)N * (size_t)K
         : fmt == QL_FMT_Q4   ? (size_t)N * (size_t)(K / 2)
                              : 2 * (size_t)N * (size_t)K;
}

size_t qlinear_scales_bytes(int64_t N, int64_t K)
{
    if (N <= 0 || K <= 0 || K % QL_BLOCK)
        return 0;
    return (size_t)N * (size_t)(K / QL_BLOCK) * 2;
}

int qlinear_quantize(int fmt, const float *W, int64_t N, int64_t K, void *codes,
                     uint16_t *scales, hipStream_t stream)
{
    if (!fmt_ok(fmt))
        return QL_ERR_INVALID;
    if (N <= 0 || K <= 0 || K % QL_BLOCK)
        return QL_ERR_SHAPE;
    if (N >= ((int64_t)1 << 40) / K)
        return QL_ERR_UNSUPPORTED;
    if (!W || !codes || !scales)
        return QL_ERR_INVALID;
    if (!aligned(W, 16) || !aligned(codes, 16) || !aligned(scales, 2))
        return QL_ERR_ALIGN;

    int *dstatus = nullptr;
    if (hipMalloc(&dstatus, sizeof(int)) != hipSuccess)
        return QL_ERR_HIP;
    int hstatus = QL_OK;
    bool ok = hipMemsetAsync(dstatus, 0, sizeof(int), stream) == hipSuccess;
    ok = ok && launch_quantize(fmt, W, N, K, (uint8_t *)codes, scales, dstatus, stream) ==
                   hipSuccess;
    ok = ok && hipMemcpyAsync(&hstatus, dstatus, sizeof(int), hipMemcpyDeviceToHost, stream) ==
                   hipSuccess;
    ok = ok && hipStreamSynchronize(stream) == hipSuccess;
    ok = hipFree(dstatus) == hipSuccess && ok;
    if (!ok)
        return QL_ERR_HIP;
    return hstatus;
}

int qlinear_forward_ep(int fmt, const void *X, int xdt, int64_t M, int64_t K, const void *codes,
                       const uint16_t *scales, int64_t N, void *Y, const ql_epilogue *ep,
                       hipStream_t stream)
{
    const ql_linear_ep l{{fmt, X, xdt, M, K, N, codes, scales, (float *)Y},
                         ep ? *ep : NO_EPILOGUE};
    const int st = check_layer(l);
    if (st != QL_OK || M == 0)
        return st;
    const ql_linear_ep *p = &l;
    WsSource src = pool_source();
    return launch_group(&p, 1, src, stream);
}

int qlinear_forward(int fmt, const void *X, int xdt, int64_t M, int64_t K, const void *codes,
                    const uint16_t *scales, int64_t N, float *Y, hipStream_t stream)
{
    return qlinear_forward_ep(fmt, X, xdt, M, K, codes, scales, N, Y, nullptr, stream);
}

int qlinear_block_forward_ep(const ql_linear_ep *lin, int n_lin, hipStream_t stream)
{
    Classes c;
    const int st = classify(lin, n_lin, c);
    if (st != QL_OK)
        return st;
    for (int k = 0; k < 6; ++k) {
        WsSource src = pool_source();
        const int s = launch_group(c.cls[k], c.cnt[k], src, stream);
        if (s != QL_OK)
            return s;
    }
    return QL_OK;
}

int qlinear_block_forward_ep_noalloc(const ql_linear_ep *lin, int n_lin, hipStream_t stream)
{
    Classes c;
    int st = classify(lin, n_lin, c);
    if (st != QL_OK)
        return st;
    uint8_t *const base = scratch_base();
    if (!base)
        return QL_ERR_HIP;
    // size every class's workspace before anything is enqueued; classes run
    // in stream order, so each reuses the scratch from its start
    WsSource dry{base, SCRATCH_BYTES, true, 0};
    for (int k = 0; k < 6; ++k)
        if ((st = launch_group(c.cls[k], c.cnt[k], dry, stream)) != QL_OK)
            return st;
    if (dry.need > SCRATCH_BYTES)
        return QL_ERR_UNSUPPORTED;
    for (int k = 0; k < 6; ++k) {
        WsSource src{base, SCRATCH_BYTES, false, 0};
        if ((st = launch_group(c.cls[k], c.cnt[k], src, stream)) != QL_OK)
            return st;
    }
    return QL_OK;
}

int qlinear_block_forward(const ql_linear *lin, int n_lin, hipStream_t stream)
{
    if (!lin || n_lin < 1 || n_lin > QL_MAX_GROUP)
        return QL_ERR_INVALID;
    ql_linear_ep l[QL_MAX_GROUP];
    for (int i = 0; i < n_lin; ++i)
        l[i] = ql_linear_ep{lin[i], NO_EPILOGUE};
    return qlinear_block_forward_ep(l, n_lin, stream);
}

int qlinear_quantize_act(const void *X, int xdt, int64_t M, int64_t K, int8_t *qx,
                         uint16_t *sx, hipStream_t stream)
{
    if (xdt != QL_DT_F32 && xdt != QL_DT_BF16)
        return QL_ERR_INVALID;
    if (M < 0 || K <= 0 || K % QL_BLOCK)
        return QL_ERR_SHAPE;
    if (M >= I31 || K >= I31)
        return QL_ERR_UNSUPPORTED;
    if (M == 0)
        return QL_OK;
    if (!X || !qx || !sx)
        return QL_ERR_INVALID;
    if (!aligned(X, 16) || !aligned(qx, 16) || !aligned(sx, 2))
        return QL_ERR_ALIGN;
    return launch_act_quant(X, xdt == QL_DT_BF16, M, K, qx, sx, stream) == hipSuccess
               ? QL_OK
               : QL_ERR_HIP;
}

int qlinear_forward_w8a8(const int8_t *qx, const uint16_t *sx, int64_t M, int64_t K,
                         const void *codes, const uint16_t *scales, int64_t N, void *Y,
                         const ql_epilogue *ep, hipStream_t stream)
{
    const ql_epilogue e = ep ? *ep : NO_EPILOGUE;
    int st = check_epilogue(e, Y);
    if (st != QL_OK)
        return st;
    if (M < 0 || N <= 0 || K <= 0 || K % QL_BLOCK)
        return QL_ERR_SHAPE;
    if (M >= I31 || N >= I31 || K >= I31)
        return QL_ERR_UNSUPPORTED;
    if (!codes || !scales || (M > 0 && (!qx || !sx || !Y)))
        return QL_ERR_INVALID;
    if (!aligned(codes, 16) || !aligned(scales, 2) ||
        (M > 0 && (!aligned(qx, 16) || !aligned(sx, 2) ||
                   !aligned(Y, e.ydt == QL_DT_BF16 ? 2 : 4))))
        return QL_ERR_ALIGN;
    if (M == 0)
        return QL_OK;
    W8Args a{};
    a.qx = qx;
    a.sx = sx;
    a.codes = (const int8_t *)codes;
    a.scales = scales;
    a.Y = (float *)Y;
    a.ep = to_epilogue(e);
    a.M = (int)M;
    a.N = (int)N;
    a.K = (int)K;
    return launch_qgemm_w8a8(a, stream) == hipSuccess ? QL_OK : QL_ERR_HIP;
}

int qlinear_steer(float *h, int64_t M, int64_t N, const float *dir, float hnorm,
                  const float *strength, hipStream_t stream)
{
    if (M < 0 || N <= 0)
        return QL_ERR_SHAPE;
    if (M >= I31 || N >= I31)
        return QL_ERR_UNSUPPORTED;
    if (!dir || !strength || (M > 0 && !h))
        return QL_ERR_INVALID;
    if (!aligned(h, 4) || !aligned(dir, 4) || !aligned(strength, 4))
        return QL_ERR_ALIGN;
    if (M == 0)
        return QL_OK;
    return launch_steer(h, M, N, dir, hnorm, strength, stream) == hipSuccess ? QL_OK
                                                                             : QL_ERR_HIP;
}

int qlinear_attention(const uint16_t *q, int64_t ldq, const uint16_t *k, int64_t ldk,
                      const uint16_t *v, int64_t ldv, int64_t B, int64_t T, int64_t H,
                      int64_t dh, float scale, void *o, int64_t ldo, int odt, hipStream_t stream)
{
    if (odt != QL_DT_F32 && odt != QL_DT_BF16)
        return QL_ERR_INVALID;
    if (B <= 0 || T <= 0 || H <= 0 || dh <= 0 || ldq < H * dh || ldk < H * dh ||
        ldv < H * dh || ldo < H * dh)
        return QL_ERR_SHAPE;
    if (dh != 64 || B * T >= I31 || B * H > 65535 || ldq >= I31 || ldk >= I31 ||
        ldv >= I31 || ldo >= I31 || (T + 127) / 128 * B * H >= I31)  // one workgroup per
        return QL_ERR_UNSUPPORTED;                                       // 128 queries
    if (!q || !k || !v || !o || !(scale >= 0.0f) || scale > 3.0e38f)
        return QL_ERR_INVALID;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || ldq % 8 || ldk % 8 ||
        ldv % 8 || !aligned(o, odt == QL_DT_BF16 ? 8 : 16) || ldo % 4)
        return QL_ERR_ALIGN;
    AttnArgs a{};
    a.q = q;
    a.k = k;
    a.v = v;
    a.ldq = ldq;
    a.ldk = ldk;
    a.ldv = ldv;
    a.o = o;
    a.ldo = ldo;
    a.B = (int)B;
    a.T = (int)T;
    a.H = (int)H;
    a.scale_log2e = (float)((double)scale * 1.4426950408889634);
    a.obf16 = odt == QL_DT_BF16 ? 1 : 0;
    return launch_attention(a, stream) == hipSuccess ? QL_OK : QL_ERR_HIP;
}

int qlinear_force_path(int path)
{
    if (path < QL_PATH_AUTO || path > QL_PATH_MID)
        return QL_ERR_INVALID;
    g_forced_path.store(path, std::memory_order_relaxed);
    return QL_OK;
}

const char *qlinear_status_string(int status)
{
    switch (status) {
    case QL_OK: return "ok";
    case QL_ERR_INVALID: return "invalid argument (null pointer, unknown enum, bad count)";
    case QL_ERR_SHAPE: return "bad shape (K must be a positive multiple of 32, N > 0, M >= 0)";
    case QL_ERR_ALIGN: return "misaligned pointer (codes/X 16 B, scales 2 B, Y 4 B)";
    case QL_ERR_RANGE: return "weights hold NaN/Inf or a block scale overflows fp16";
    case QL_ERR_UNSUPPORTED: return "size beyond what the kernels index";
    case QL_ERR_HIP: return "HIP runtime or launch failure";
    default: return "unknown status";
    }
}

}  // extern "C"
