// Stack executor: a network's conv layers validated and planned once, then
// enqueued back to back, or captured into one HIP graph and replayed.
//
// Batch-1 inference (the setting of the paper's latency tables, Sec. 4.2)
// runs layers of a few microseconds each, so per-call host work and launch
// gaps matter as much as the kernels.  The executor resolves every layer's
// kernel and split-K plan up front, owns one split-K workspace sized for the
// largest layer (layers run in stream order, so they can share it), and can
// record the whole pass -- optionally repeated `steps` times, with an event
// before every kernel launch -- as a graph that replays with a single launch.
//
// On request (miconv_stack_overlap), layers that do not depend on each other
// overlap in the untimed graph: at create the executor derives every layer's
// dependencies from the address ranges it reads and writes (read after
// write, write after write, write after read), and a layer whose successor
// does not depend on it is put on a second stream (ResNet's projection
// shortcut runs beside the first two convs of its block).  Cross-stream
// dependencies become event waits, which under capture are graph edges; each
// pass forks the second stream from the first at its start and joins it at
// its end, and the two streams use separate halves of the workspace.  Eager
// and timed passes stay in one stream, in layer order.  Measured on MI355X,
// the edges cost more than the overlap gains (ResNet-50 at batch 1: 0.400 ms
// in one stream, 0.494 ms overlapped; batch 64 bf16: 1.52 against 1.55 ms),
// so it is off by default.
#include "../../include/miconv.h"
#include "internal.h"

#include <cstdio>

#include <algorithm>
#include <new>
#include <string>
#include <vector>

struct miconv_stack {
    int device = 0;
    std::vector<miconv::Resolved> layers;
    std::vector<int> launch_layer;          // layer of every kernel launch of one pass
    std::vector<std::string> launch_name;   // its kernel name
    float *partials = nullptr;              // split-K workspace shared by all layers
    std::vector<void *> packed;             // packed copies of filters, made at create
    bool stamps = false;                    // events are (start, end) pairs per launch
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    std::vector<hipEvent_t> events;         // steps * launches + 1 when timed
    int steps = 0;
    // two-stream schedule of the untimed graph
    std::vector<int> sid;                   // stream of every layer (0: the caller's, 1: side)
    std::vector<std::vector<int>> cross;    // earlier layers on the other stream it waits for
    std::vector<hipEvent_t> done;           // recorded after a layer another stream waits for
    size_t ws_half = 0;                     // bytes of workspace per stream
    hipStream_t side = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
    bool overlap = false;
};

using namespace miconv;

namespace {

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

void drop_graph(miconv_stack *s)
{
    if (s->exec) hipGraphExecDestroy(s->exec);
    if (s->graph) hipGraphDestroy(s->graph);
    for (hipEvent_t e : s->events) hipEventDestroy(e);
    s->exec = nullptr;
    s->graph = nullptr;
    s->events.clear();
    s->stamps = false;
    s->steps = 0;
}

// Record an event.  Under capture a plain record only marks a capture
// dependency, so an event-record node is added to the graph by hand, after
// the nodes the stream currently depends on, and becomes the new dependency.
hipError_t record(hipEvent_t ev, hipStream_t st)
{
    hipStreamCaptureStatus status = hipStreamCaptureStatusNone;
    unsigned long long id = 0;
    hipGraph_t g = nullptr;
    const hipGraphNode_t *deps = nullptr;
    size_t ndeps = 0;
    hipError_t e = hipStreamGetCaptureInfo_v2(st, &status, &id, &g, &deps, &ndeps);
    if (e != hipSuccess) return e;
    if (status != hipStreamCaptureStatusActive) return hipEventRecord(ev, st);
    hipGraphNode_t node = nullptr;
    e = hipGraphAddEventRecordNode(&node, g, deps, ndeps, ev);
    if (e != hipSuccess) return e;
    return hipStreamUpdateCaptureDependencies(st, &node, 1, hipStreamSetCaptureDependencies);
}

struct EventCursor {
    hipEvent_t *next;
};

hipError_t record_next(void *ctx, hipStream_t st)
{
    EventCursor *c = static_cast<EventCursor *>(ctx);
    return record(*c->next++, st);
}

// Eager kernel timing: the next launch gets the next two events as its
// start/end stamps (the runtime writes the kernel's own execution interval).
hipError_t arm_next(void *ctx, hipStream_t)
{
    EventCursor *c = static_cast<EventCursor *>(ctx);
    t_launch_start = *c->next++;
    t_launch_stop = *c->next++;
    return hipSuccess;
}

// One pass over every layer; with `ev`, an event before every kernel launch
// (or, `stamps`, a start and an end event stamped on every kernel launch).
hipError_t enqueue_all(miconv_stack *s, hipStream_t st, hipEvent_t *ev, bool stamps = false)
{
    EventCursor cur{ev};
    LaunchHook hook{stamps ? arm_next : record_next, &cur};
    for (size_t i = 0; i < s->layers.size(); ++i) {
        hipError_t e = enqueue(s->layers[i], s->partials, st, ev ? &hook : nullptr);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// One pass on two streams (see the file comment); st is the caller's.
hipError_t enqueue_two_streams(miconv_stack *s, hipStream_t st)
{
    hipStream_t sts[2] = {st, s->side};
    hipError_t e;
    if ((e = hipEventRecord(s->fork, st)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(s->side, s->fork, 0)) != hipSuccess) return e;
    for (size_t i = 0; i < s->layers.size(); ++i) {
        const int k = s->sid[i];
        for (int j : s->cross[i])
            if ((e = hipStreamWaitEvent(sts[k], s->done[j], 0)) != hipSuccess) return e;
        float *ws = s->partials ? reinterpret_cast<float *>(reinterpret_cast<char *>(s->partials) + k * s->ws_half)
                                : nullptr;
        if ((e = enqueue(s->layers[i], ws, sts[k])) != hipSuccess) return e;
        if (s->done[i] && (e = hipEventRecord(s->done[i], sts[k])) != hipSuccess) return e;
    }
    if ((e = hipEventRecord(s->join, s->side)) != hipSuccess) return e;
    return hipStreamWaitEvent(st, s->join, 0);
}

// Byte range [lo, hi) of a layer's input, output and residual.
struct Span {
    uintptr_t lo = 0, hi = 0;
    bool overlaps(const Span &o) const { return lo < o.hi && o.lo < hi; }
};

void layer_spans(const Resolved &r, Span *x, Span *y, Span *res)
{
    const ConvProblem &p = r.p;
    const long out = (long)p.K * p.P * p.Q;
    const long img = p.ysn > out ? p.ysn : out;
    const long yn = (long)(p.N - 1) * img + out;
    const long xe = r.kind == OP_DENSE_BF16 || r.kind == OP_MAXPOOL_BF16_NHWC ? 2 : 4;   // bytes per element
    const long ye = p.ycl ? 2 : 4;
    x->lo = (uintptr_t)r.x;
    x->hi = x->lo + (uintptr_t)((long)p.N * p.C * p.H * p.W * xe);
    y->lo = (uintptr_t)r.y;
    y->hi = y->lo + (uintptr_t)(yn * ye);
    res->lo = (uintptr_t)p.res;
    res->hi = p.res ? res->lo + (uintptr_t)(yn * ye) : res->lo;
}

// Dependencies and the two-stream assignment (called once, at create).
int plan_streams(miconv_stack *s)
{
    const size_t n = s->layers.size();
    std::vector<Span> xs(n), ys(n), rs(n);
    for (size_t i = 0; i < n; ++i) layer_spans(s->layers[i], &xs[i], &ys[i], &rs[i]);
    auto depends = [&](size_t i, size_t j) {   // layer i (later) on layer j
        const bool reads_j = xs[i].overlaps(ys[j]) || rs[i].overlaps(ys[j]);
        const bool overwrites = ys[i].overlaps(ys[j]) || ys[i].overlaps(xs[j]) || ys[i].overlaps(rs[j]);
        return reads_j || overwrites;
    };
    s->sid.assign(n, 0);
    s->cross.assign(n, {});
    s->done.assign(n, nullptr);
    bool any = false;
    for (size_t i = 0; i + 1 < n; ++i)
        if (!depends(i + 1, i) && (i == 0 || s->sid[i - 1] == 0)) {
            s->sid[i] = 1;
            any = true;
        }
    if (!any) {
        s->sid.clear();
        return MICONV_OK;
    }
    for (size_t i = 0; i < n; ++i)
        for (size_t j = 0; j < i; ++j)
            if (s->sid[j] != s->sid[i] && depends(i, j)) s->cross[i].push_back((int)j);
    for (size_t i = 0; i < n; ++i)
        for (int j : s->cross[i])
            if (!s->done[j]) {
                hipError_t e = hipEventCreateWithFlags(&s->done[j], hipEventDisableTiming);
                if (e != hipSuccess) return set_hip_error(e);
            }
    hipError_t e = hipStreamCreateWithFlags(&s->side, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s->fork, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s->join, hipEventDisableTiming);
    return e == hipSuccess ? MICONV_OK : set_hip_error(e);
}

int make_events(miconv_stack *s, int steps, bool stamps = false)
{
    const size_t per = s->launch_layer.size();
    s->events.resize(stamps ? 2 * (size_t)steps * per : (size_t)steps * per + 1, nullptr);
    s->stamps = stamps;
    for (auto &ev : s->events) {
        hipError_t e = hipEventCreate(&ev);
        if (e != hipSuccess) {
            ev = nullptr;
            drop_graph(s);
            return set_hip_error(e);
        }
    }
    return MICONV_OK;
}

int capture_on(miconv_stack *s, int steps, int timed, hipStream_t st)
{
    drop_graph(s);
    const size_t n = s->launch_layer.size();
    if (timed) {
        int rc = make_events(s, steps);
        if (rc != MICONV_OK) return rc;
    }
    hipError_t e = hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
        drop_graph(s);
        return set_hip_error(e);
    }
    for (int k = 0; k < steps && e == hipSuccess; ++k)
        e = !timed && s->overlap && !s->sid.empty() ? enqueue_two_streams(s, st)
                                      : enqueue_all(s, st, timed ? &s->events[(size_t)k * n] : nullptr);
    if (e == hipSuccess && timed) e = record(s->events.back(), st);
    hipGraph_t g = nullptr;
    hipError_t e2 = hipStreamEndCapture(st, &g);
    s->graph = g;
    if (e == hipSuccess) e = e2;
    if (e == hipSuccess) e = hipGraphInstantiate(&s->exec, s->graph, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        drop_graph(s);
        return set_hip_error(e);
    }
    s->steps = steps;
    return MICONV_OK;
}

}  // namespace

extern "C" {

int miconv_stack_create(const miconv_conv_desc *layers, int n, miconv_stack **out)
{
    if (!out) return MICONV_ERR_NULL;
    *out = nullptr;
    if (n <= 0) return MICONV_ERR_SHAPE;
    if (!layers) return MICONV_ERR_NULL;
    miconv_stack *s = new (std::nothrow) miconv_stack;
    if (!s) return MICONV_ERR_HIP;
    hipError_t e = hipGetDevice(&s->device);
    if (e != hipSuccess) {
        delete s;
        return set_hip_error(e);
    }
    size_t need_p = 0;
    for (int i = 0; i < n; ++i) {
        const miconv_conv_desc &d = layers[i];
        Resolved r;
        int rc = resolve(d.op, MICONV_ALGO_AUTO, MODE_SCRATCH | MODE_PREPACK, d.N, d.C, d.H, d.W, d.K, d.R,
                         d.S, d.stride, d.pad, d.groups, d.x, d.w, d.bias, static_cast<float *>(d.y), d.relu,
                         &r, d.layout);
        if (rc == MICONV_OK) rc = set_output_stride(r, d.y_image_stride);
        if (rc == MICONV_OK) rc = set_residual(r, static_cast<const float *>(d.res));
        if (rc != MICONV_OK) {
            miconv_stack_destroy(s);
            return rc;
        }
        if (r.wlayout != WL_GIVEN) {
            // Pre-computing: pack the filters once, in the layout the kernel
            // reads, for every replay.
            void *pk = nullptr;
            e = hipMalloc(&pk, packed_bytes(r));
            if (e == hipSuccess) s->packed.push_back(pk);
            if (e == hipSuccess) e = launch_pack(r, pk, nullptr);
            if (e != hipSuccess) {
                miconv_stack_destroy(s);
                return set_hip_error(e);
            }
            set_packed(r, pk);
        }
        need_p = std::max(need_p, round_up(workspace_bytes(r), 256));
        s->layers.push_back(r);
        char buf[512];
        int launches = 0;
        describe(r, buf, sizeof buf, &launches);
        std::string names(buf);
        for (int j = 0; j < launches; ++j) {
            const size_t cut = names.find(" + ");
            s->launch_layer.push_back(i);
            s->launch_name.push_back(names.substr(0, cut));
            names = cut == std::string::npos ? std::string() : names.substr(cut + 3);
        }
    }
    int rc = plan_streams(s);
    if (rc != MICONV_OK) {
        miconv_stack_destroy(s);
        return rc;
    }
    s->ws_half = need_p;
    if (need_p) {
        void *ptr = nullptr;
        e = hipMalloc(&ptr, s->sid.empty() ? need_p : 2 * need_p);
        if (e != hipSuccess) {
            miconv_stack_destroy(s);
            return set_hip_error(e);
        }
        s->partials = static_cast<float *>(ptr);
    }
    if (!s->packed.empty()) {
        e = hipStreamSynchronize(nullptr);   // packs run on the default stream
        if (e != hipSuccess) {
            miconv_stack_destroy(s);
            return set_hip_error(e);
        }
    }
    *out = s;
    return MICONV_OK;
}

int miconv_stack_size(const miconv_stack *s)
{
    return s ? (int)s->layers.size() : MICONV_ERR_NULL;
}

int miconv_stack_describe(const miconv_stack *s, int layer, char *buf, int buflen)
{
    if (!s || !buf || buflen <= 0) return MICONV_ERR_NULL;
    if (layer < 0 || layer >= (int)s->layers.size()) return MICONV_ERR_SHAPE;
    int launches = 0;
    describe(s->layers[layer], buf, buflen, &launches);
    return launches;
}

int miconv_stack_launches(const miconv_stack *s)
{
    return s ? (int)s->launch_layer.size() : MICONV_ERR_NULL;
}

int miconv_stack_launch_info(const miconv_stack *s, int launch, char *buf, int buflen)
{
    if (!s || !buf || buflen <= 0) return MICONV_ERR_NULL;
    if (launch < 0 || launch >= (int)s->launch_layer.size()) return MICONV_ERR_SHAPE;
    snprintf(buf, buflen, "%s", s->launch_name[launch].c_str());
    return s->launch_layer[launch];
}

int miconv_stack_launch(miconv_stack *s, void *stream)
{
    if (!s) return MICONV_ERR_NULL;
    hipError_t e = enqueue_all(s, static_cast<hipStream_t>(stream), nullptr);
    return e == hipSuccess ? MICONV_OK : set_hip_error(e);
}

int miconv_stack_launch_timed(miconv_stack *s, int steps, void *stream)
{
    if (!s) return MICONV_ERR_NULL;
    if (steps < 1) return MICONV_ERR_SHAPE;
    drop_graph(s);
    const size_t n = s->launch_layer.size();
    int rc = make_events(s, steps, true);
    if (rc != MICONV_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    for (int k = 0; k < steps && e == hipSuccess; ++k)
        e = enqueue_all(s, st, &s->events[2 * (size_t)k * n], true);
    t_launch_start = t_launch_stop = nullptr;
    if (e != hipSuccess) {
        drop_graph(s);
        return set_hip_error(e);
    }
    s->steps = steps;
    return MICONV_OK;
}

int miconv_stack_overlap(miconv_stack *s, int enable)
{
    if (!s) return MICONV_ERR_NULL;
    s->overlap = enable != 0;
    if (!s->overlap) return 0;
    int side = 0;
    for (int k : s->sid) side += k;
    return side;
}

int miconv_stack_capture(miconv_stack *s, int steps, int timed, void *stream)
{
    if (!s) return MICONV_ERR_NULL;
    if (steps < 1) return MICONV_ERR_SHAPE;
    // The legacy default stream cannot be captured; record on a private stream
    // instead (the graph can still be launched on any stream).
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipStream_t tmp = nullptr;
    if (!st) {
        hipError_t e = hipStreamCreateWithFlags(&tmp, hipStreamNonBlocking);
        if (e != hipSuccess) return set_hip_error(e);
        st = tmp;
    }
    const int rc = capture_on(s, steps, timed, st);
    if (tmp) hipStreamDestroy(tmp);
    return rc;
}

int miconv_stack_replay(miconv_stack *s, void *stream)
{
    if (!s) return MICONV_ERR_NULL;
    if (!s->exec) return MICONV_ERR_UNSUPPORTED;
    hipError_t e = hipGraphLaunch(s->exec, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? MICONV_OK : set_hip_error(e);
}

int miconv_stack_times(const miconv_stack *s, float *ms, long capacity)
{
    if (!s || !ms) return MICONV_ERR_NULL;
    if (s->events.empty()) return MICONV_ERR_UNSUPPORTED;
    const size_t total = s->stamps ? s->events.size() / 2 : s->events.size() - 1;
    if ((size_t)capacity < total) return MICONV_ERR_SHAPE;
    for (size_t i = 0; i < total; ++i) {
        hipError_t e = s->stamps ? hipEventElapsedTime(&ms[i], s->events[2 * i], s->events[2 * i + 1])
                                 : hipEventElapsedTime(&ms[i], s->events[i], s->events[i + 1]);
        if (e != hipSuccess) return set_hip_error(e);
    }
    return MICONV_OK;
}

int miconv_stack_destroy(miconv_stack *s)
{
    if (!s) return MICONV_OK;
    drop_graph(s);
    if (s->partials) hipFree(s->partials);
    for (void *p : s->packed) hipFree(p);
    for (hipEvent_t ev : s->done)
        if (ev) hipEventDestroy(ev);
    if (s->fork) hipEventDestroy(s->fork);
    if (s->join) hipEventDestroy(s->join);
    if (s->side) hipStreamDestroy(s->side);
    delete s;
    return MICONV_OK;
}

}  // extern "C"
