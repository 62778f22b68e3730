// Executor: validates the call, resolves symbolic buffers to device pointers
// and enqueues the plan's launches on the caller's stream.  No host
// synchronisation, no device allocation.
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "capi_internal.h"
#include "kernels.h"
#include "plan.h"

namespace ce {
namespace {

struct Ptrs {
    const void* const* in;
    void* out;
    const void* dout;
    void* const* din;
    void* ws;
};

void* resolve(const BufRef& b, const Ptrs& P) {
    void* base = nullptr;
    switch (b.kind) {
        case BUF_IN: base = const_cast<void*>(P.in[b.index]); break;
        case BUF_OUT: base = P.out; break;
        case BUF_DOUT: base = const_cast<void*>(P.dout); break;
        case BUF_DIN: base = P.din ? P.din[b.index] : nullptr; break;
        case BUF_WS: base = (char*)P.ws + b.offset; break;
        default: return nullptr;
    }
    // a view that starts inside the buffer (phases of a strided transposed conv)
    return base ? (void*)((char*)base + b.shift) : nullptr;
}

hipError_t raw_launch(const Launch& ln, const Ptrs& P, hipStream_t s) {
    const void* a = resolve(ln.a, P);
    const void* b = resolve(ln.b, P);
    void* c = resolve(ln.c, P);
    void* d = resolve(ln.d, P);
    int variant = ln.kind & 0xff;
    switch (variant) {
        case K_GENERIC_THREAD:
        case K_GENERIC_WAVE:
        case K_GENERIC_BLOCK: return launch_generic(ln, a, b, c, s);
        case K_CP_FWD: {
            const void* ops[5] = {a, b, resolve(ln.extra[0], P), resolve(ln.extra[1], P),
                                  resolve(ln.extra[2], P)};
            return launch_cp_fwd(ln, ops, c, s);
        }
        case K_TT_FWD:
        case K_TT_PREP: {
            const void* ops[4] = {a, b, resolve(ln.extra[0], P), resolve(ln.extra[1], P)};
            return launch_tt_fwd(ln, ops, c, s);
        }
        case K_RCP_FWD: {
            const void* ops[5] = {a, b, resolve(ln.extra[0], P), resolve(ln.extra[1], P),
                                  resolve(ln.extra[2], P)};
            return launch_rcp_fwd(ln, ops, c, s);
        }
        case K_RCP_BWD: {
            const void* ops[12] = {a, b};
            for (int i = 0; i < 10; i++) ops[2 + i] = resolve(ln.extra[i], P);
            return launch_rcp_bwd(ln, ops, s);
        }
        case K_RCP_PREP: {
            const void* ops[5];
            for (int i = 0; i < 5; i++) ops[i] = resolve(ln.extra[i], P);
            return launch_rcp_prep(ln, ops, s);
        }
        case K_CP_BWD: {
            const void* ops[11] = {a, b, c};
            for (int i = 0; i < 8; i++) ops[3 + i] = resolve(ln.extra[i], P);
            return launch_cp_bwd(ln, ops, s);
        }
        case K_GPAIR: return launch_gpair(ln, a, b, c, resolve(ln.extra[0], P), d, s);
        case K_REDUCE_MULTI: {
            const void* parts[4] = {};
            void* outs[4] = {};
            for (size_t j = 0; j < 4 && 2 * j + 1 < ln.extra.size(); j++) {
                parts[j] = resolve(ln.extra[2 * j], P);
                outs[j] = resolve(ln.extra[2 * j + 1], P);
            }
            return launch_reduce_multi(ln, parts, outs, s);
        }
        default: return launch_fast(ln, a, b, c, d, s);
    }
}

// ---- launch timing ---------------------------------------------------------
struct TimingRec {
    hipEvent_t a, b;
    const Launch* ln;
    std::string kname, what;
    float ms = 0;
    double bytes = 0, flops = 0;
};
thread_local bool g_timing = false;
thread_local std::string g_only;   // record only this kernel label (empty: all)
thread_local std::vector<TimingRec> g_recs;
thread_local std::vector<hipEvent_t> g_pool;
thread_local size_t g_pool_used = 0;

hipEvent_t next_event() {
    if (g_pool_used == g_pool.size()) {
        hipEvent_t ev;
        if (hipEventCreate(&ev) != hipSuccess) fail(CE_ERR_HIP, "hipEventCreate failed");
        g_pool.push_back(ev);
    }
    return g_pool[g_pool_used++];
}

void check_ws(const ce_plan* p, size_t need, void* ws, size_t ws_bytes) {
    if (ws_bytes < need)
        fail(CE_ERR_WORKSPACE, "workspace of " + std::to_string(ws_bytes) + " B < required " +
                                   std::to_string(need) + " B");
    if (need && !ws) fail(CE_ERR_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)ws) & 255) fail(CE_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    (void)p;
}

hipError_t run_launch(const Launch& ln, const Ptrs& P, hipStream_t s) {
    if (!g_timing || (!g_only.empty() && ln.kname != g_only)) return raw_launch(ln, P, s);
    TimingRec r;
    r.a = next_event();
    r.b = next_event();
    r.ln = &ln;
    r.kname = ln.kname;
    r.what = ln.what;
    r.bytes = ln.alg_bytes;
    r.flops = ln.alg_flops;
    hipError_t e = hipEventRecord(r.a, s);
    if (e != hipSuccess) return e;
    e = raw_launch(ln, P, s);
    if (e != hipSuccess) return e;
    e = hipEventRecord(r.b, s);
    if (e == hipSuccess) g_recs.push_back(r);
    return e;
}

}  // namespace
}  // namespace ce

using namespace ce;

extern "C" ce_status ce_timing_begin(void) { return ce_timing_begin_kernel(nullptr); }

extern "C" ce_status ce_timing_begin_kernel(const char* kernel) {
    return guard([&] {
        g_recs.clear();
        g_pool_used = 0;
        g_only = kernel ? kernel : "";
        g_timing = true;
    });
}

extern "C" ce_status ce_timing_end(int* n_records) {
    return guard([&] {
        g_timing = false;
        if (!g_recs.empty()) {
            hipError_t e = hipEventSynchronize(g_recs.back().b);
            if (e != hipSuccess) fail(CE_ERR_HIP, std::string("hipEventSynchronize: ") + hipGetErrorString(e));
            for (auto& r : g_recs) {
                e = hipEventElapsedTime(&r.ms, r.a, r.b);
                if (e != hipSuccess) fail(CE_ERR_HIP, std::string("hipEventElapsedTime: ") + hipGetErrorString(e));
            }
        }
        if (n_records) *n_records = (int)g_recs.size();
    });
}

extern "C" ce_status ce_timing_record(int i, const char** kernel, const char** step, float* ms,
                                      double* bytes, double* flops) {
    return guard([&] {
        if (i < 0 || i >= (int)g_recs.size()) fail(CE_ERR_ARG, "record index out of range");
        const TimingRec& r = g_recs[i];
        if (kernel) *kernel = r.kname.c_str();
        if (step) *step = r.what.c_str();
        if (ms) *ms = r.ms;
        if (bytes) *bytes = r.bytes;
        if (flops) *flops = r.flops;
    });
}

extern "C" ce_status ce_forward(const ce_plan* p, const void* const* in, void* out, void* ws,
                                size_t ws_bytes, ce_stream stream) {
    return guard([&] {
        if (!p || !in || !out) fail(CE_ERR_ARG, "NULL plan, inputs or output");
        if (!p->executable) fail(CE_ERR_UNSUPPORTED, p->why_not);
        for (int i = 0; i < p->e.n; i++)
            if (!in[i]) fail(CE_ERR_ARG, "input " + std::to_string(i) + " is NULL");
        check_ws(p, p->ws_fwd, ws, ws_bytes);
        Ptrs P{in, out, nullptr, nullptr, ws};
        hipStream_t s = (hipStream_t)stream;
        for (const Launch& ln : p->fwd) {
            hipError_t err = run_launch(ln, P, s);
            if (err != hipSuccess)
                fail(CE_ERR_HIP, std::string("kernel launch failed (") + ln.what + "): " +
                                     hipGetErrorString(err));
        }
    });
}

namespace ce {
namespace {

// Checks of a backward call; returns the bitmask of wanted gradients.
uint32_t check_backward(const ce_plan* p, const void* const* in, const void* dout, void* const* din) {
    if (!p || !in || !dout || !din) fail(CE_ERR_ARG, "NULL plan, inputs, dout or din");
    if (!p->executable) fail(CE_ERR_UNSUPPORTED, p->why_not);
    uint32_t wanted = 0;
    for (int i = 0; i < p->e.n; i++) {
        if (!in[i]) fail(CE_ERR_ARG, "input " + std::to_string(i) + " is NULL");
        if (din[i]) wanted |= 1u << i;
    }
    return wanted;
}

void run_backward(const ce_plan* p, const void* const* in, const void* dout, void* const* din,
                  uint32_t wanted, void* ws, hipStream_t s) {
    if (!wanted) return;
    Ptrs P{in, nullptr, dout, din, ws};
    for (const Launch& ln : p->bwd) {
        if (ln.need && !(ln.need & wanted)) continue;
        hipError_t err = run_launch(ln, P, s);
        if (err != hipSuccess)
            fail(CE_ERR_HIP, std::string("kernel launch failed (") + ln.what + "): " +
                                 hipGetErrorString(err));
    }
}

// ---- workspace of the allocation-free backward ------------------------------
// A fixed device array (one copy on every GPU the library's code object is
// loaded on, held until the process ends).  Host code never uses the array's
// name as an address: its device address is looked up once per device, with
// that device current, and kept in scratch_addr.
static __device__ __align__(256) unsigned char scratch[CE_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on the first
// call on that device).
void* scratch_addr(hipStream_t s) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) fail(CE_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) fail(CE_ERR_UNSUPPORTED, "device index beyond 63");
    if (s) {
        int sdev = -1;
        e = hipStreamGetDevice(s, &sdev);
        if (e != hipSuccess) fail(CE_ERR_HIP, std::string("hipStreamGetDevice: ") + hipGetErrorString(e));
        if (sdev != dev) fail(CE_ERR_ARG, "the stream belongs to another device than the current one");
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            fail(CE_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_addr[dev] = ptr;
    }
    return g_scratch_addr[dev];
}

}  // namespace
}  // namespace ce

extern "C" ce_status ce_backward(const ce_plan* p, const void* const* in, const void* dout,
                                 void* const* din, void* ws, size_t ws_bytes, ce_stream stream) {
    return guard([&] {
        const uint32_t wanted = check_backward(p, in, dout, din);
        check_ws(p, p->ws_bwd, ws, ws_bytes);
        run_backward(p, in, dout, din, wanted, ws, (hipStream_t)stream);
    });
}

extern "C" ce_status ce_backward_noalloc(const ce_plan* p, const void* const* in, const void* dout,
                                         void* const* din, ce_stream stream) {
    return guard([&] {
        const uint32_t wanted = check_backward(p, in, dout, din);
        if (p->save_mask)
            fail(CE_ERR_UNSUPPORTED, "the plan's backward reads intermediates from the forward's workspace");
        if (p->ws_bwd > (size_t)CE_NOALLOC_WORKSPACE_BYTES)
            fail(CE_ERR_WORKSPACE, "the backward needs " + std::to_string(p->ws_bwd) +
                                       " B of workspace, more than the " +
                                       std::to_string((size_t)CE_NOALLOC_WORKSPACE_BYTES) +
                                       " B the allocation-free entry point holds");
        hipStream_t s = (hipStream_t)stream;
        void* ws = scratch_addr(s);
        run_backward(p, in, dout, din, wanted, ws, s);
    });
}
