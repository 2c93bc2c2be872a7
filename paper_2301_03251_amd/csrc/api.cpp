// api.cpp -- the C ABI (qlayer.h): validation, workspace layout, launch order.
//
// One call = angle binding, then either one whole-state launch (small n) or
// the forward tile passes, a fused pass (last forward pass + <Z> partials +
// lambda seed + first backward pass), the remaining backward passes in reverse
// order, and the final reductions -- all on the caller's stream, no host
// synchronisation, no device allocation.
#include "qlayer.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "launch.hpp"
#include "plan.hpp"

using namespace qlayer;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Device tables of one dtype's plan, packed into one blob that each call
// copies into the head of the workspace.
struct Tables {
    std::vector<uint8_t> blob;
    size_t off_pass = 0, off_phase = 0, off_ops = 0, off_gslot = 0, off_slots = 0;
    size_t off_xptr = 0, off_xslot = 0, off_wptr = 0, off_wslot = 0, off_gates = 0, off_diag = 0;
    size_t off_fuse = 0, off_czg = 0, off_pthr = 0;
    size_t off_pptr = 0, off_pops = 0;  // product-prefix CSR (per qubit)
    std::vector<DevPass> passes;
    int n_diags = 0, n_fuses = 0;
    int n_ops = 0;
    int bwd_first = 0;
};

template <typename T>
size_t put(std::vector<uint8_t>& blob, const std::vector<T>& v) {
    size_t off = align256(blob.size());
    blob.resize(off + std::max<size_t>(sizeof(T) * v.size(), 16), 0);
    if (!v.empty()) std::memcpy(blob.data() + off, v.data(), sizeof(T) * v.size());
    return off;
}

void build_tables(const Circuit& c, int dt, Tables& T) {
    const Plan& pl = c.plan[dt];
    std::vector<DevPass> passes;
    std::vector<DevOp> ops;
    std::vector<int32_t> gsl;
    if (!pl.whole_state) {
        for (const PassPlan& pp : pl.passes) {
            DevPass d{};
            d.k = pl.k;
            d.log_t = pl.log_t;
            uint64_t in_tile = 0;
            for (int j = 0; j < pl.k; j++) {
                d.tile_qubit[j] = pp.qubits[j];
                in_tile |= 1ull << pp.qubits[j];
            }
            for (int q = 0; q < c.n; q++)
                if (!(in_tile >> q & 1)) d.fixed_qubit[d.n_fixed++] = q;
            d.fwd_begin = (int)ops.size();
            ops.insert(ops.end(), pp.fwd_ops.begin(), pp.fwd_ops.end());
            d.fwd_end = (int)ops.size();
            d.load_phase = pp.first_phase;
            d.bwd_phase = pp.last_phase;
            d.gslot_base = (int)gsl.size();
            gsl.insert(gsl.end(), pp.gslots.begin(), pp.gslots.end());
            d.n_gslots = (int)pp.gslots.size();
            d.n_exchanges = pp.n_transposes;
            d.index = (int)passes.size();
            passes.push_back(d);
        }
        // backward ranges after every forward range (the binding kernel gives
        // ops from bwd_first on the inverse rotation)
        T.bwd_first = (int)ops.size();
        for (size_t p = 0; p < pl.passes.size(); p++) {
            passes[p].bwd_begin = (int)ops.size();
            ops.insert(ops.end(), pl.passes[p].bwd_ops.begin(), pl.passes[p].bwd_ops.end());
            passes[p].bwd_end = (int)ops.size();
        }
    }
    std::vector<SlotSrc> slots;
    for (const Slot& sl : c.slots) slots.push_back({sl.src, sl.index, sl.scale, sl.c1, sl.c2, sl.c3});
    std::vector<int32_t> xptr(c.n_inputs + 1, 0), wptr(c.n_weights + 1, 0), xs, ws;
    for (int f = 0; f < c.n_inputs; f++) {
        for (int s = 0; s < (int)slots.size(); s++)
            if (slots[s].src == S_INPUT && slots[s].index == f) xs.push_back(s);
        xptr[f + 1] = (int)xs.size();
    }
    for (int p = 0; p < c.n_weights; p++) {
        for (int s = 0; s < (int)slots.size(); s++)
            if (slots[s].src == S_WEIGHT && slots[s].index == p) ws.push_back(s);
        wptr[p + 1] = (int)ws.size();
    }
    std::vector<DevGate> gates;
    for (const Gate& g : c.gates) gates.push_back({g.kind, g.q0, g.q1, g.slot});

    T.blob.clear();
    T.off_pass = put(T.blob, passes);
    T.off_phase = put(T.blob, pl.phases);
    T.off_ops = put(T.blob, ops);
    T.off_gslot = put(T.blob, gsl);
    T.off_slots = put(T.blob, slots);
    T.off_xptr = put(T.blob, xptr);
    T.off_xslot = put(T.blob, xs);
    T.off_wptr = put(T.blob, wptr);
    T.off_wslot = put(T.blob, ws);
    T.off_gates = put(T.blob, gates);
    T.off_diag = put(T.blob, pl.diags);
    T.n_diags = (int)pl.diags.size();
    T.off_fuse = put(T.blob, pl.fuses);
    T.n_fuses = (int)pl.fuses.size();
    T.off_czg = put(T.blob, pl.czgs);
    // per phase, the thread-index part of every thread's layout: tile bits
    // (low PTHR_TB_BITS bits) and LDS byte offset (above), one word per lane
    // for the lane bits, one per wavefront index for the higher thread bits;
    // a thread's layout is its two words XORed
    std::vector<uint32_t> pthr;
    if (!pl.whole_state) {
        pthr.reserve(pl.phases.size() * PTHR_WORDS);
        for (const DevPhase& F : pl.phases)
            for (int e = 0; e < PTHR_WORDS; e++) {
                const int b0 = e < 64 ? 0 : 6, nb = e < 64 ? std::min(6, pl.log_t) : std::max(0, pl.log_t - 6);
                const uint32_t v = e < 64 ? (uint32_t)e : (uint32_t)(e - 64);
                uint32_t tb = 0, ts = 0;
                for (int i = 0; i < nb; i++)
                    if (v >> i & 1u) {
                        tb |= 1u << F.thr_bit[b0 + i];
                        ts ^= F.thr_slot[b0 + i];
                    }
                pthr.push_back(tb | ts << PTHR_TB_BITS);
            }
    }
    T.off_pthr = put(T.blob, pthr);
    T.off_pptr = put(T.blob, pl.pre_ptr);
    T.off_pops = put(T.blob, pl.pre_ops);
    T.blob.resize(align256(T.blob.size()), 0);
    T.passes = passes;
    T.n_ops = (int)ops.size();
}

struct Layout {
    size_t tables = 0, coef = 0, opc = 0, dzc = 0, fzc = 0, zpart = 0, gpart = 0, psi = 0, lam = 0, total = 0;
    size_t enorm = 0, edot = 0;  // embedding: per-circuit |x| or basis index; L_b
    size_t keep = 0;             // kept forward states: n_keep buffers of state_bytes each
    size_t phi = 0, env = 0;     // product prefix: per-circuit factors; per-tile environment sums
    size_t state_bytes = 0;
    int n_keep = 0;
    int n_wg = 1;
};

bool mul_ok(size_t a, size_t b, size_t& out) {
    if (a != 0 && b > SIZE_MAX / a) return false;
    out = a * b;
    return true;
}

}  // namespace

struct ql_circuit {
    Circuit c;
    Tables t[2];
    // pinned host copies of the table blobs (made on the first call of each
    // dtype), so the per-call upload is an asynchronous DMA
    void* pinned[2] = {nullptr, nullptr};
    std::once_flag pin_once[2];
    // an event per stream that copied from a pinned blob, recorded after each
    // such copy: destruction waits for these copies only
    std::mutex up_mu;
    std::vector<std::pair<hipStream_t, hipEvent_t>> uploads;
    // timing
    int timing = 0;
    struct Ev {
        hipEvent_t a, b;
        int cls;
    };
    std::vector<Ev> ev;
    size_t ev_used = 0;
};

namespace {

// own_psi = false: the caller's state buffer holds psi (ql_state), so the
// workspace has none.
int compute_layout(const ql_circuit* h, int dt, int64_t B, int mode, Layout& L, bool own_psi = true) {
    const Circuit& c = h->c;
    const Plan& pl = c.plan[dt];
    const size_t amp = dt == 0 ? 8 : 16;
    if (B < 1) return fail(QL_EINVAL, "batch must be >= 1");
    if (B > (int64_t)1 << 30) return fail(QL_EINVAL, "batch too large");
    const int maxq = dt == 0 ? QL_MAX_QUBITS_C64 : QL_MAX_QUBITS_C128;
    if (c.n > maxq) return fail(QL_EUNSUPPORTED, "too many qubits for this dtype");
    L = Layout{};
    if (pl.whole_state) {
        L.n_wg = 1;
    } else {
        const int64_t tiles = (int64_t)1 << (c.n - pl.k);
        // Default: about 8192 workgroups per launch, each looping over a few
        // tiles. Two workgroups share a CU; with few long-lived workgroups
        // their load, compute and store phases overlap worse (30 qubits, one
        // sample: 229 ms per step at 512 workgroups, 211 at 2048, 204 at
        // 8192, 206 at 32768). At most half a sample's tiles, so that the
        // two-tile forward mode gives every workgroup a pair.
        int64_t nwg = c.opts.wg_per_sample ? c.opts.wg_per_sample : (8192 + B - 1) / B;
        const int64_t cap = c.opts.wg_per_sample ? tiles : std::max<int64_t>(1, tiles / 2);
        nwg = std::max<int64_t>(1, std::min<int64_t>(nwg, cap));
        if (nwg * B > (int64_t)INT32_MAX) return fail(QL_ENOMEM, "grid too large");
        L.n_wg = (int)nwg;
    }
    const bool bwd = mode == QL_MODE_FWD_BWD || mode == QL_MODE_FWD_BWD_KEEP;
    size_t off = 0, sz = 0;
    L.tables = off;
    off = align256(off + h->t[dt].blob.size());
    L.coef = off;
    if (!mul_ok((size_t)B * (size_t)std::max(1, (int)c.slots.size()), amp, sz)) return fail(QL_ENOMEM, "size overflow");
    off = align256(off + sz);
    if (!pl.whole_state) {
        // per-sample op records (16 bytes fp32 / 32 bytes fp64) plus an end record
        L.opc = off;
        if (!mul_ok((size_t)B * (size_t)(h->t[dt].n_ops + 1), dt == 0 ? 16 : 32, sz))
            return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
        // per-sample phase tables of the RZ groups
        L.dzc = off;
        if (!mul_ok((size_t)B * (size_t)h->t[dt].n_diags, (size_t)DZ_REGS * amp, sz))
            return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
        // per-sample RZ coefficients of the RY-RZ pair ops
        L.fzc = off;
        if (!mul_ok((size_t)B * (size_t)h->t[dt].n_fuses, amp, sz)) return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
    }
    L.zpart = off;
    if (!mul_ok((size_t)B * (size_t)L.n_wg, (size_t)c.n * 8, sz)) return fail(QL_ENOMEM, "size overflow");
    off = align256(off + sz);
    if (pl.product) {
        // per circuit and qubit the prefix factor (phi(0), phi(1)), complex fp64
        L.phi = off;
        if (!mul_ok((size_t)B, (size_t)c.n * 32, sz)) return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
    }
    if (bwd) {
        L.gpart = off;
        if (!mul_ok((size_t)B * (size_t)L.n_wg, (size_t)std::max(1, (int)c.slots.size()) * 8, sz))
            return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
    }
    if (bwd && pl.product) {
        // per sample, environment workgroup and qubit: (re, im) of r_q(0) and r_q(1), fp64
        L.env = off;
        if (!mul_ok((size_t)B * (size_t)env_workgroups(dt, c.n, B), (size_t)c.n * 32, sz))
            return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
    }
    // state buffers: psi between tile passes or for an embedded initial state
    // (the caller's buffer when own_psi is false); lambda between backward
    // passes or for the amplitude-embedding gradient (lambda_0). Keep mode
    // gives each forward pass but the last its own output buffer, which the
    // backward pass over the next pass reads instead of a stored
    // un-computed state.
    const bool multi = !pl.whole_state && pl.passes.size() > 1;
    const bool emb = c.embed != E_NONE, amp_bwd = bwd && c.embed == E_AMPLITUDE;
    const bool keep = multi && mode == QL_MODE_FWD_BWD_KEEP;
    // the product prefix's environment reads lambda at the end of the backward sweep
    const bool need_psi = own_psi && (emb || (multi && !keep));
    const bool need_lam = (bwd && multi) || amp_bwd || (bwd && !pl.whole_state && pl.product);
    size_t st = 0;
    if (need_psi || need_lam || keep)
        if (!mul_ok((size_t)B, ((size_t)1 << c.n) * amp, st)) return fail(QL_ENOMEM, "size overflow");
    L.state_bytes = st;
    if (need_psi) {
        L.psi = off;
        off = align256(off + st);
    }
    if (need_lam) {
        L.lam = off;
        off = align256(off + st);
    }
    if (keep) {
        L.keep = off;
        L.n_keep = (int)pl.passes.size() - 1;
        if (!mul_ok(st, (size_t)L.n_keep, sz) || sz > SIZE_MAX - off - 256)
            return fail(QL_ENOMEM, "size overflow");
        off = align256(off + sz);
    }
    if (emb) {
        L.enorm = off;
        off = align256(off + (size_t)B * 8);
    }
    if (amp_bwd) {
        L.edot = off;
        off = align256(off + (size_t)B * 8);
    }
    L.total = off;
    return QL_OK;
}

// Scratch of ql_forward_backward_static: one copy on every GPU the library
// runs on, held until the process ends. In host code `scratch` names a
// host-side stand-in, not device memory: only the address hipGetSymbolAddress
// returns (per device, with that device current) is passed to kernels.
__device__ __align__(256) unsigned char scratch[QL_STATIC_SCRATCH_BYTES];
std::mutex g_scratch_mu;
std::map<int, void*> g_scratch;

// The current device's scratch address (looked up once per device).
int static_scratch(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(QL_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch.find(dev);
    if (it == g_scratch.end()) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(QL_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        it = g_scratch.emplace(dev, p).first;
    }
    *out = it->second;
    return QL_OK;
}

std::mutex g_dev_mu;
std::set<int> g_dev_ready;
size_t g_lds_limit = 65536;

int ensure_device() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(QL_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if (g_dev_ready.count(dev)) return QL_OK;
    int optin = 0;
    if (hipDeviceGetAttribute(&optin, hipDeviceAttributeSharedMemPerBlockOptin, dev) != hipSuccess || optin <= 0)
        optin = 65536;
    e = configure_kernels((size_t)optin);
    if (e != hipSuccess) return fail(QL_EHIP, std::string("hipFuncSetAttribute: ") + hipGetErrorString(e));
    g_lds_limit = (size_t)optin;
    g_dev_ready.insert(dev);
    return QL_OK;
}

struct Timer {
    ql_circuit* h;
    hipStream_t s;
    int cls = 0;
    bool on = false;
    void start(int c) {
        cls = c;
        on = h && (h->timing >> c & 1) != 0;
        if (!on) return;
        if (h->ev_used == h->ev.size()) {
            ql_circuit::Ev e{};
            if (hipEventCreate(&e.a) != hipSuccess || hipEventCreate(&e.b) != hipSuccess) return;
            h->ev.push_back(e);
        }
        h->ev[h->ev_used].cls = c;
        (void)hipEventRecord(h->ev[h->ev_used].a, s);
    }
    void stop() {
        if (!on || h->ev_used >= h->ev.size()) return;
        (void)hipEventRecord(h->ev[h->ev_used].b, s);
        h->ev_used++;
    }
};

// One call's device context: the plan tables of its dtype, the workspace
// layout and the stream.
struct Ctx {
    ql_circuit* h;
    int dt;
    const Circuit& c;
    const Plan& pl;
    const Tables& T;
    uint8_t* W;
    Layout L;
    hipStream_t stream;
    Timer tm;
    bool no_alloc = false;  // make no host or device allocation (no pinned copy, no event)
    // the angle sources of the current circuits (set by bind(); the
    // one-wavefront kernel binds the angles itself)
    const void* inputs = nullptr;
    const void* weights = nullptr;
    int64_t v0 = 0;
    int32_t vper = 0;
};

int upload_tables(Ctx& x) {
    if (x.no_alloc) {  // from the handle's own (pageable) copy
        hipError_t e = hipMemcpyAsync(x.W + x.L.tables, x.T.blob.data(), x.T.blob.size(), hipMemcpyHostToDevice,
                                      x.stream);
        return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("table upload: ") + hipGetErrorString(e));
    }
    std::call_once(x.h->pin_once[x.dt], [&] {
        void* p = nullptr;
        if (hipHostMalloc(&p, x.T.blob.size(), hipHostMallocDefault) == hipSuccess) {
            std::memcpy(p, x.T.blob.data(), x.T.blob.size());
            x.h->pinned[x.dt] = p;
        } else {
            (void)hipGetLastError();  // keep the pageable copy
        }
    });
    const void* src = x.h->pinned[x.dt] ? x.h->pinned[x.dt] : (const void*)x.T.blob.data();
    hipError_t e = hipMemcpyAsync(x.W + x.L.tables, src, x.T.blob.size(), hipMemcpyHostToDevice, x.stream);
    if (e != hipSuccess) return fail(QL_EHIP, std::string("table upload: ") + hipGetErrorString(e));
    if (!x.h->pinned[x.dt]) return QL_OK;
    // mark the copy's completion on this stream for ql_circuit_destroy
    std::lock_guard<std::mutex> lk(x.h->up_mu);
    hipEvent_t ev = nullptr;
    for (auto& u : x.h->uploads)
        if (u.first == x.stream) ev = u.second;
    if (!ev) {
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) return fail(QL_EHIP, std::string("hipEventCreate: ") + hipGetErrorString(e));
        x.h->uploads.push_back({x.stream, ev});
    }
    e = hipEventRecord(ev, x.stream);
    return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
}

// Arguments of the product-prefix kernels for B circuits of this call.
PrefixArgs prefix_args(const Ctx& x, int64_t B) {
    PrefixArgs pa{};
    pa.inputs = x.inputs;
    pa.weights = x.weights;
    pa.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
    pa.pre_ptr = (const int32_t*)(x.W + x.L.tables + x.T.off_pptr);
    pa.pre_ops = (const DevPrefix*)(x.W + x.L.tables + x.T.off_pops);
    pa.phi = (double*)(x.W + x.L.phi);
    pa.lam = x.L.lam ? (const void*)(x.W + x.L.lam) : nullptr;
    pa.envpart = x.L.env ? (double*)(x.W + x.L.env) : nullptr;
    pa.gpart = x.L.gpart ? (double*)(x.W + x.L.gpart) : nullptr;
    pa.B = B;
    pa.n = x.c.n;
    pa.F = x.c.n_inputs;
    pa.n_wg = x.L.n_wg;
    pa.env_wg = env_workgroups(x.dt, x.c.n, B);
    return pa;
}

// Angle binding for B circuits. With vper > 0 the circuits are the shifted
// copies of a parameter-shift chunk: circuit i is virtual circuit v = v0 + i,
// sample v / vper, and v % vper = 2s+1 (2s+2) shifts rotation slot s by
// +pi/2 (-pi/2).
int bind(Ctx& x, int64_t B, const void* inputs, const void* weights, int64_t v0, int32_t vper, bool bwd) {
    hipError_t e;
    x.inputs = inputs;
    x.weights = weights;
    x.v0 = v0;
    x.vper = vper;
    if (x.pl.whole_state && whole_uses_wave(x.c.n, bwd, B)) return QL_OK;  // bound in the kernel
    if (x.pl.whole_state) {
        BindArgs ba{};
        ba.inputs = inputs;
        ba.weights = weights;
        ba.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
        ba.coef = x.W + x.L.coef;
        ba.B = B;
        ba.n_slots = (int)x.c.slots.size();
        ba.F = x.c.n_inputs;
        ba.v0 = v0;
        ba.vper = vper;
        x.tm.start(2);
        e = launch_bind(x.dt, ba, x.stream);
        x.tm.stop();
    } else {
        BindTileArgs ba{};
        ba.inputs = inputs;
        ba.weights = weights;
        ba.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
        ba.ops = (const DevOp*)(x.W + x.L.tables + x.T.off_ops);
        ba.opc = x.W + x.L.opc;
        ba.diags = (const DevDiag*)(x.W + x.L.tables + x.T.off_diag);
        ba.dzc = x.W + x.L.dzc;
        ba.n_diags = x.T.n_diags;
        ba.fuses = (const DevFuse*)(x.W + x.L.tables + x.T.off_fuse);
        ba.fzc = x.W + x.L.fzc;
        ba.n_fuses = x.T.n_fuses;
        ba.B = B;
        ba.n_ops = x.T.n_ops;
        ba.bwd_first = x.T.bwd_first;
        ba.F = x.c.n_inputs;
        ba.v0 = v0;
        ba.vper = vper;
        x.tm.start(2);
        e = launch_bind_tile(x.dt, ba, x.stream);
        if (e == hipSuccess && x.pl.product) {
            PrefixArgs pa = prefix_args(x, B);
            pa.v0 = v0;
            pa.vper = vper;
            e = launch_bind_prefix(x.dt, pa, x.stream);
        }
        x.tm.stop();
    }
    return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("k_bind: ") + hipGetErrorString(e));
}

// Initial states of B circuits for an embedding (into psi: the caller's state
// buffer or the workspace's). Circuit i is sample i, or sample (v0 + i) / vper
// of a parameter-shift chunk.
int embed(Ctx& x, int64_t B, const void* inputs, void* psi, int64_t v0, int32_t vper) {
    if (x.c.embed == E_NONE) return QL_OK;
    EmbedArgs ea{};
    ea.inputs = inputs;
    ea.psi = psi;
    ea.norm = (double*)(x.W + x.L.enorm);
    ea.count = B;
    ea.v0 = v0;
    ea.vper = vper;
    ea.kind = x.c.embed;
    ea.first = x.c.embed_first;
    ea.F = x.c.n_inputs;
    ea.n = x.c.n;
    x.tm.start(2);
    hipError_t e = launch_embed(x.dt, ea, x.stream);
    x.tm.stop();
    return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("k_embed: ") + hipGetErrorString(e));
}

// The state passes of B circuits: the whole-state kernel, or the forward tile
// passes, the fused pass and (bwd) the backward passes. Writes the <Z> partials
// (and, bwd, the gradient partials) of the workspace.
int state_passes(Ctx& x, int64_t B, bool bwd, const void* grad_out, void* psi_ext = nullptr) {
    const Circuit& c = x.c;
    const Plan& pl = x.pl;
    const size_t amp = x.dt == 0 ? 8 : 16;
    double* zpart = (double*)(x.W + x.L.zpart);
    double* gpart = bwd ? (double*)(x.W + x.L.gpart) : nullptr;
    // an embedded initial state is in the state buffer (written by embed())
    const bool emb = c.embed != E_NONE, amp_bwd = bwd && c.embed == E_AMPLITUDE;
    void* psi_buf = psi_ext ? psi_ext : (x.L.psi ? (void*)(x.W + x.L.psi) : nullptr);
    // keep mode: kept[p] is the state after forward pass p
    const bool keep = bwd && x.L.n_keep > 0;
    auto kept = [&](int p) -> void* { return x.W + x.L.keep + (size_t)p * x.L.state_bytes; };
    if (pl.whole_state) {
        WholeArgs wa{};
        wa.gates = (const DevGate*)(x.W + x.L.tables + x.T.off_gates);
        wa.n_gates = (int)c.gates.size();
        wa.n = c.n;
        wa.n_slots = (int)c.slots.size();
        wa.bwd = bwd ? 1 : 0;
        wa.B = B;
        wa.coef = x.W + x.L.coef;
        wa.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
        wa.inputs = x.inputs;
        wa.weights = x.weights;
        wa.F = c.n_inputs;
        wa.v0 = x.v0;
        wa.vper = x.vper;
        wa.grad_out = grad_out;
        wa.zpart = zpart;
        wa.gpart = gpart;
        wa.psi_out = psi_ext;
        wa.psi_in = emb ? psi_buf : nullptr;
        wa.lam_out = amp_bwd ? (void*)(x.W + x.L.lam) : nullptr;
        const int dim = 1 << c.n;
        const int threads = std::max(64, std::min(256, dim / 4));
        const size_t lds = 2 * (size_t)dim * amp + (size_t)c.n * (threads / 64) * 8 + 64;
        if (lds > g_lds_limit) return fail(QL_EUNSUPPORTED, "state does not fit in LDS");
        x.tm.start(1);
        hipError_t e = launch_whole(x.dt, wa, threads, lds, x.stream);
        x.tm.stop();
        return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("k_whole: ") + hipGetErrorString(e));
    }
    const int m = (int)pl.passes.size();
    const int threads = 1 << pl.log_t;
    const int NW = threads / 64;
    // psi_in: the state the pass loads; psi_out: where it stores its state
    auto launch_pass = [&](int p, int flags, void* psi_in, void* psi_out) -> int {
        const DevPass& d = x.T.passes[p];
        TileArgs ta{};
        ta.psi = psi_in;
        ta.psi_out = psi_out;
        ta.lam = x.L.lam ? (void*)(x.W + x.L.lam) : nullptr;
        ta.pass = (const DevPass*)(x.W + x.L.tables + x.T.off_pass) + p;
        ta.phases = (const DevPhase*)(x.W + x.L.tables + x.T.off_phase);
        ta.ops = (const DevOp*)(x.W + x.L.tables + x.T.off_ops);
        ta.gslots = (const int32_t*)(x.W + x.L.tables + x.T.off_gslot) + d.gslot_base;
        ta.opc = x.W + x.L.opc;
        ta.dzc = x.W + x.L.dzc;
        ta.n_diags = x.T.n_diags;
        ta.fzc = x.W + x.L.fzc;
        ta.n_fuses = x.T.n_fuses;
        ta.czg = (const DevCzg*)(x.W + x.L.tables + x.T.off_czg);
        ta.pthr = (const uint32_t*)(x.W + x.L.tables + x.T.off_pthr);
        ta.grad_out = grad_out;
        ta.zpart = zpart;
        ta.gpart = gpart;
        ta.B = B;
        ta.tiles = (int64_t)1 << (c.n - pl.k);
        ta.n = c.n;
        ta.n_ops = x.T.n_ops;
        ta.n_wg = x.L.n_wg;
        ta.flags = flags;
        ta.n_gslots = (flags & PF_BWD) ? d.n_gslots : 0;
        ta.phi = pl.product ? (const double*)(x.W + x.L.phi) : nullptr;
        // dynamic LDS: <Z> scratch and gradient accumulators (the exchange
        // buffer is static)
        const size_t st = tile_static_lds(x.dt, pl.log_r, threads), real = x.dt == 0 ? 4 : 8;
        const size_t lds = (size_t)c.n * NW * 8 + (size_t)ta.n_gslots * NW * TILE_GRAD_WORDS * real;
        if (lds + st > g_lds_limit)
            return fail(QL_EUNSUPPORTED, "tile pass needs more LDS than available");
        x.tm.start(0);
        hipError_t le = launch_tile(x.dt, pl.log_r, (flags & PF_BWD) != 0, ta, threads, lds, x.stream);
        x.tm.stop();
        if (le != hipSuccess) return fail(QL_EHIP, std::string("k_tile: ") + hipGetErrorString(le));
        return QL_OK;
    };
    int rc;
    // the first pass starts from |0...0> (or the product state of the prefix
    // factors) in registers unless an embedding wrote the initial state; the
    // last backward pass stores lambda_0 when the amplitude-embedding gradient
    // or the product prefix's environment needs it
    const int init = emb ? 0 : (pl.product ? PF_PRODUCT : PF_INIT);
    const int lam0 = (amp_bwd || pl.product) ? PF_STORE_LAM : 0;
    for (int p = 0; p + 1 < m; p++) {
        void* out = keep ? kept(p) : psi_buf;
        void* in = keep && p > 0 ? kept(p - 1) : (p == 0 && !emb ? out : psi_buf);
        rc = launch_pass(p, (p == 0 ? init : 0) | PF_FWD | PF_STORE_PSI, in, out);
        if (rc) return rc;
    }
    // with kept states no backward pass stores psi: the next one loads the
    // forward state instead
    const int bwd_psi = keep ? 0 : PF_STORE_PSI;
    int last = (m == 1 ? init : 0) | PF_FWD | (psi_ext ? PF_STORE_PSI : PF_ZPART);
    if (bwd) last |= PF_SEED | PF_BWD | (m > 1 ? (bwd_psi | PF_STORE_LAM) : lam0);
    void* last_in = keep ? kept(m - 2) : psi_buf;
    rc = launch_pass(m - 1, last, last_in, keep ? last_in : psi_buf);
    if (rc) return rc;
    if (bwd)
        for (int p = m - 2; p >= 0; p--) {
            void* in = keep ? kept(p) : psi_buf;
            rc = launch_pass(p, PF_LOAD_LAM | PF_BWD | (p > 0 ? (bwd_psi | PF_STORE_LAM) : lam0), in, in);
            if (rc) return rc;
        }
    return QL_OK;
}

// Final fixed-order reductions of the partials into expz (and gradients).
int reduce(Ctx& x, int64_t B, bool grads, void* expz, void* grad_inputs, void* grad_weights) {
    ReduceArgs ra{};
    ra.zpart = (const double*)(x.W + x.L.zpart);
    ra.gpart = grads ? (const double*)(x.W + x.L.gpart) : nullptr;
    ra.expz = expz;
    ra.grad_inputs = grad_inputs;
    ra.grad_weights = grad_weights;
    ra.x_ptr = (const int32_t*)(x.W + x.L.tables + x.T.off_xptr);
    ra.x_slot = (const int32_t*)(x.W + x.L.tables + x.T.off_xslot);
    ra.w_ptr = (const int32_t*)(x.W + x.L.tables + x.T.off_wptr);
    ra.w_slot = (const int32_t*)(x.W + x.L.tables + x.T.off_wslot);
    ra.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
    ra.B = B;
    ra.n = x.c.n;
    ra.n_wg = x.L.n_wg;
    ra.F = x.c.n_inputs;
    ra.P = x.c.n_weights;
    ra.n_slots = (int)x.c.slots.size();
    ra.grads = grads ? 1 : 0;
    x.tm.start(3);
    hipError_t e = launch_reduce(x.dt, ra, x.stream);
    x.tm.stop();
    return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("k_reduce: ") + hipGetErrorString(e));
}

int check_args(const Circuit& c, const void* inputs, const void* weights, const void* expz, bool need_g,
               const void* grad_out, const void* ws) {
    if (!expz) return fail(QL_EINVAL, "expz is NULL");
    if (c.n_inputs > 0 && !inputs) return fail(QL_EINVAL, "inputs is NULL");
    if (c.n_weights > 0 && !weights) return fail(QL_EINVAL, "weights is NULL");
    if (need_g && !grad_out) return fail(QL_EINVAL, "grad_out is NULL");
    if (!ws) return fail(QL_EINVAL, "workspace is NULL");
    return QL_OK;
}

int run(const ql_circuit* hc, ql_dtype dtype, int64_t B, int mode, const void* inputs,
        const void* weights, const void* grad_out, void* expz, void* grad_inputs,
        void* grad_weights, void* ws, size_t ws_bytes, hipStream_t stream, bool no_alloc = false) {
    if (!hc) return fail(QL_EINVAL, "circuit is NULL");
    ql_circuit* h = const_cast<ql_circuit*>(hc);  // only the timing state is touched
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    const int dt = (int)dtype;
    const bool bwd = mode == QL_MODE_FWD_BWD;
    Layout L;
    int rc = compute_layout(h, dt, B, mode, L);
    if (rc) return rc;
    if (bwd) {  // keep the forward states when the workspace holds them
        Layout K;
        if (compute_layout(h, dt, B, QL_MODE_FWD_BWD_KEEP, K) == QL_OK && K.n_keep > 0 && ws_bytes >= K.total)
            L = K;
    }
    rc = check_args(h->c, inputs, weights, expz, bwd, grad_out, ws);
    if (rc) return rc;
    if (ws_bytes < L.total)
        return fail(QL_ENOMEM, "workspace too small: need " + std::to_string(L.total) + " bytes, got " +
                                   std::to_string(ws_bytes));
    rc = ensure_device();
    if (rc) return rc;
    Ctx x{h, dt, h->c, h->c.plan[dt], h->t[dt], (uint8_t*)ws, L, stream, Timer{h, stream}};
    x.no_alloc = no_alloc;
    if (no_alloc) x.tm.h = nullptr;  // no timing events either
    if ((rc = upload_tables(x))) return rc;
    if ((rc = bind(x, B, inputs, weights, 0, 0, bwd))) return rc;
    if ((rc = embed(x, B, inputs, x.L.psi ? (void*)(x.W + x.L.psi) : nullptr, 0, 0))) return rc;
    if ((rc = state_passes(x, B, bwd, grad_out))) return rc;
    if (bwd && x.pl.product) {  // the prefix rotations' gradient terms, into gpart
        const PrefixArgs pa = prefix_args(x, B);
        x.tm.start(3);
        hipError_t e = launch_env(dt, pa, stream);
        if (e == hipSuccess) e = launch_env_grad(dt, pa, stream);
        x.tm.stop();
        if (e != hipSuccess) return fail(QL_EHIP, std::string("k_env: ") + hipGetErrorString(e));
    }
    if ((rc = reduce(x, B, bwd, expz, grad_inputs, grad_weights))) return rc;
    if (bwd && grad_inputs && h->c.embed == E_AMPLITUDE) {
        EmbedGradArgs ga{};
        ga.inputs = inputs;
        ga.lam = x.W + x.L.lam;
        ga.norm = (const double*)(x.W + x.L.enorm);
        ga.dot = (double*)(x.W + x.L.edot);
        ga.grad_inputs = grad_inputs;
        ga.B = B;
        ga.first = h->c.embed_first;
        ga.F = h->c.n_inputs;
        ga.n = h->c.n;
        x.tm.start(3);
        hipError_t e = launch_embed_grad(dt, ga, stream);
        x.tm.stop();
        if (e != hipSuccess) return fail(QL_EHIP, std::string("k_embed_grad: ") + hipGetErrorString(e));
    }
    return QL_OK;
}

// Workspace of a parameter-shift call: the forward layout of one chunk of
// C shifted circuits, then the chunk's <Z> values [C][n] (Real) and the VJP
// of every shifted circuit [B * (2S+1)] (fp64).
struct ShiftLayout {
    Layout L;
    int64_t chunk = 0, total = 0;
    size_t ev = 0, dv = 0, bytes = 0;
};

int shift_layout(const ql_circuit* h, int dt, int64_t B, int64_t max_chunk, ShiftLayout& S) {
    if (B < 1) return fail(QL_EINVAL, "batch must be >= 1");
    if (max_chunk < 0) return fail(QL_EINVAL, "max_chunk must be >= 0");
    const int64_t V = 2 * (int64_t)h->c.n_param_slots + 1;
    if (B > ((int64_t)1 << 40) / V) return fail(QL_EINVAL, "batch too large");
    S.total = B * V;
    S.chunk = max_chunk > 0 ? std::min<int64_t>(max_chunk, S.total) : S.total;
    int rc = compute_layout(h, dt, S.chunk, QL_MODE_FWD, S.L);
    if (rc) return rc;
    const size_t real = dt == 0 ? 4 : 8;
    size_t off = S.L.total, sz;
    S.ev = off;
    if (!mul_ok((size_t)S.chunk, (size_t)h->c.n * real, sz)) return fail(QL_ENOMEM, "size overflow");
    off = align256(off + sz);
    S.dv = off;
    if (!mul_ok((size_t)S.total, 8, sz)) return fail(QL_ENOMEM, "size overflow");
    S.bytes = align256(off + sz);
    return QL_OK;
}

int param_shift(const ql_circuit* hc, ql_dtype dtype, int64_t B, const void* inputs,
                const void* weights, const void* grad_out, void* expz, void* grad_inputs,
                void* grad_weights, int64_t max_chunk, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (!hc) return fail(QL_EINVAL, "circuit is NULL");
    ql_circuit* h = const_cast<ql_circuit*>(hc);
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    const int dt = (int)dtype;
    ShiftLayout S;
    int rc = shift_layout(h, dt, B, max_chunk, S);
    if (rc) return rc;
    rc = check_args(h->c, inputs, weights, expz, true, grad_out, ws);
    if (rc) return rc;
    if (grad_inputs && h->c.embed == E_AMPLITUDE)
        return fail(QL_EUNSUPPORTED, "parameter shift gives no gradient for amplitude-embedded features "
                                     "(pass grad_inputs = NULL, or use ql_forward_backward)");
    if (ws_bytes < S.bytes)
        return fail(QL_ENOMEM, "workspace too small: need " + std::to_string(S.bytes) + " bytes, got " +
                                   std::to_string(ws_bytes));
    rc = ensure_device();
    if (rc) return rc;
    Ctx x{h, dt, h->c, h->c.plan[dt], h->t[dt], (uint8_t*)ws, S.L, stream, Timer{h, stream}};
    if ((rc = upload_tables(x))) return rc;
    const int32_t V = (int32_t)(2 * h->c.n_param_slots + 1);
    void* ev = x.W + S.ev;
    double* dv = (double*)(x.W + S.dv);
    for (int64_t v0 = 0; v0 < S.total; v0 += S.chunk) {
        const int64_t cb = std::min(S.chunk, S.total - v0);
        if ((rc = bind(x, cb, inputs, weights, v0, V, false))) return rc;
        if ((rc = embed(x, cb, inputs, x.L.psi ? (void*)(x.W + x.L.psi) : nullptr, v0, V))) return rc;
        if ((rc = state_passes(x, cb, false, nullptr))) return rc;
        if ((rc = reduce(x, cb, false, ev, nullptr, nullptr))) return rc;
        ShiftDotArgs sa{};
        sa.ev = ev;
        sa.grad_out = grad_out;
        sa.expz = expz;
        sa.dv = dv;
        sa.v0 = v0;
        sa.count = cb;
        sa.vper = V;
        sa.n = h->c.n;
        x.tm.start(3);
        hipError_t e = launch_shift_dot(dt, sa, stream);
        x.tm.stop();
        if (e != hipSuccess) return fail(QL_EHIP, std::string("k_shift_dot: ") + hipGetErrorString(e));
    }
    ShiftGradArgs ga{};
    ga.dv = dv;
    ga.grad_inputs = grad_inputs;
    ga.grad_weights = grad_weights;
    ga.x_ptr = (const int32_t*)(x.W + x.L.tables + x.T.off_xptr);
    ga.x_slot = (const int32_t*)(x.W + x.L.tables + x.T.off_xslot);
    ga.w_ptr = (const int32_t*)(x.W + x.L.tables + x.T.off_wptr);
    ga.w_slot = (const int32_t*)(x.W + x.L.tables + x.T.off_wslot);
    ga.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
    ga.B = B;
    ga.vper = V;
    ga.F = h->c.n_inputs;
    ga.P = h->c.n_weights;
    x.tm.start(3);
    hipError_t e = launch_shift_grad(dt, ga, stream);
    x.tm.stop();
    return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("k_shift_grad: ") + hipGetErrorString(e));
}

int state(const ql_circuit* hc, ql_dtype dtype, int64_t B, const void* inputs, const void* weights,
          void* psi, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (!hc) return fail(QL_EINVAL, "circuit is NULL");
    ql_circuit* h = const_cast<ql_circuit*>(hc);
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    const int dt = (int)dtype;
    Layout L;
    int rc = compute_layout(h, dt, B, QL_MODE_FWD, L, false);
    if (rc) return rc;
    if (!psi) return fail(QL_EINVAL, "psi is NULL");
    rc = check_args(h->c, inputs, weights, psi, false, nullptr, ws);
    if (rc) return rc;
    if (ws_bytes < L.total)
        return fail(QL_ENOMEM, "workspace too small: need " + std::to_string(L.total) + " bytes, got " +
                                   std::to_string(ws_bytes));
    rc = ensure_device();
    if (rc) return rc;
    Ctx x{h, dt, h->c, h->c.plan[dt], h->t[dt], (uint8_t*)ws, L, stream, Timer{h, stream}};
    if ((rc = upload_tables(x))) return rc;
    if ((rc = bind(x, B, inputs, weights, 0, 0, false))) return rc;
    if ((rc = embed(x, B, inputs, psi, 0, 0))) return rc;
    if ((rc = state_passes(x, B, false, nullptr, psi))) return rc;
    if (x.pl.whole_state) return QL_OK;  // exact gates: no phase to undo
    BindTileArgs ba{};
    ba.inputs = inputs;
    ba.weights = weights;
    ba.slots = (const SlotSrc*)(x.W + x.L.tables + x.T.off_slots);
    ba.ops = (const DevOp*)(x.W + x.L.tables + x.T.off_ops);
    ba.diags = (const DevDiag*)(x.W + x.L.tables + x.T.off_diag);
    ba.n_diags = x.T.n_diags;
    ba.fuses = (const DevFuse*)(x.W + x.L.tables + x.T.off_fuse);
    ba.n_fuses = x.T.n_fuses;
    ba.B = B;
    ba.n_ops = x.T.n_ops;
    ba.bwd_first = x.T.bwd_first;
    ba.F = h->c.n_inputs;
    hipError_t e = launch_state_phase(dt, ba, (double*)(x.W + x.L.zpart), psi, h->c.n, stream);
    return e == hipSuccess ? QL_OK : fail(QL_EHIP, std::string("state phase: ") + hipGetErrorString(e));
}

// Blocks of 2^bb amplitudes for shot sampling.
int sample_blocks(int n, int& bb, int64_t& nblk) {
    if (n < 1 || n > QL_MAX_QUBITS_C64) return fail(QL_EINVAL, "n_qubits out of range [1, 32]");
    bb = std::min(n, 12);
    nblk = (int64_t)1 << (n - bb);
    return QL_OK;
}

int sample_bytes(int n, int64_t B, size_t& out) {
    int bb;
    int64_t nblk;
    int rc = sample_blocks(n, bb, nblk);
    if (rc) return rc;
    if (B < 1) return fail(QL_EINVAL, "batch must be >= 1");
    // block prefix, then the 64 lane-chunk sums of every block
    size_t chunks = 0;
    if (!mul_ok((size_t)B, (size_t)nblk * 8, out) || !mul_ok(out, 64, chunks))
        return fail(QL_ENOMEM, "size overflow");
    out = align256(out) + chunks;
    return QL_OK;
}

Options to_options(const ql_options* o) {
    Options r;
    if (o) {
        r.log_regs = o->log_regs;
        r.log_threads = o->log_threads;
        r.low_qubits = o->low_qubits;
        r.max_gates_per_pass = o->max_gates_per_pass;
        r.force_tiled = o->force_tiled;
        r.wg_per_sample = o->wg_per_sample;
        r.rz_groups = o->rz_groups;
        r.pass_search = o->pass_search;
        r.product_prefix = o->product_prefix;
        r.cz_groups = o->cz_groups;
    }
    return r;
}

}  // namespace

extern "C" {

int ql_circuit_create_desc(int32_t n_qubits, const ql_gate* gates, int32_t n_gates, int32_t n_inputs,
                           int32_t n_weights, const ql_circuit_desc* desc, const ql_options* opts,
                           ql_circuit** out) {
    if (!out) return fail(QL_EINVAL, "out is NULL");
    *out = nullptr;
    static_assert(sizeof(ql_gate) == 5 * sizeof(int32_t), "ql_gate layout");
    static_assert(QL_CRX == P_CRX && QL_CRY == P_CRY && QL_CRZ == P_CRZ && QL_PAULI == P_PAULI, "kinds");
    static_assert(QL_EMBED_BASIS == E_BASIS && QL_EMBED_AMPLITUDE == E_AMPLITUDE, "embeddings");
    Extras ext;
    if (desc) {
        ext.embed = desc->embedding;
        ext.embed_first = desc->embed_first;
        ext.pauli_p = desc->pauli_p;
    }
    ql_circuit* h = new (std::nothrow) ql_circuit();
    if (!h) return fail(QL_ENOMEM, "host allocation failed");
    std::string err;
    try {
        err = build_circuit(n_qubits, (const int32_t*)gates, n_gates, n_inputs, n_weights, ext,
                            to_options(opts), h->c);
        if (err.empty())
            for (int dt = 0; dt < 2; dt++) build_tables(h->c, dt, h->t[dt]);
    } catch (const std::bad_alloc&) {
        delete h;
        return fail(QL_ENOMEM, "host allocation failed");
    }
    if (!err.empty()) {
        delete h;
        return fail(err.compare(0, 7, "option:") == 0 ? QL_EUNSUPPORTED : QL_EINVAL, err);
    }
    *out = h;
    g_err.clear();
    return QL_OK;
}

int ql_circuit_create_ex(int32_t n_qubits, const ql_gate* gates, int32_t n_gates, int32_t n_inputs,
                         int32_t n_weights, const ql_options* opts, ql_circuit** out) {
    return ql_circuit_create_desc(n_qubits, gates, n_gates, n_inputs, n_weights, nullptr, opts, out);
}

int ql_circuit_create(int32_t n_qubits, const ql_gate* gates, int32_t n_gates, int32_t n_inputs,
                      int32_t n_weights, ql_circuit** out) {
    return ql_circuit_create_desc(n_qubits, gates, n_gates, n_inputs, n_weights, nullptr, nullptr, out);
}

void ql_circuit_destroy(ql_circuit* h) {
    if (!h) return;
    // table uploads of calls still queued read the pinned copies: wait for
    // the last one on each stream that made any (not for the whole device)
    for (auto& u : h->uploads) {
        (void)hipEventSynchronize(u.second);
        (void)hipEventDestroy(u.second);
    }
    for (void* p : h->pinned)
        if (p) (void)hipHostFree(p);
    for (auto& e : h->ev) {
        (void)hipEventDestroy(e.a);
        (void)hipEventDestroy(e.b);
    }
    delete h;
}

int ql_workspace_bytes(const ql_circuit* h, ql_dtype dtype, int64_t batch, int mode, size_t* out) {
    if (!h || !out) return fail(QL_EINVAL, "NULL argument");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    if (mode != QL_MODE_FWD && mode != QL_MODE_FWD_BWD && mode != QL_MODE_FWD_BWD_KEEP)
        return fail(QL_EINVAL, "unknown mode");
    Layout L;
    int rc = compute_layout(h, (int)dtype, batch, mode, L);
    if (rc) return rc;
    *out = L.total;
    return QL_OK;
}

int ql_forward(const ql_circuit* h, ql_dtype dtype, int64_t batch, const void* inputs,
               const void* weights, void* expz, void* ws, size_t ws_bytes, hipStream_t stream) {
    int rc = run(h, dtype, batch, QL_MODE_FWD, inputs, weights, nullptr, expz, nullptr, nullptr, ws,
                 ws_bytes, stream);
    if (rc == QL_OK) g_err.clear();
    return rc;
}

int ql_forward_backward(const ql_circuit* h, ql_dtype dtype, int64_t batch, const void* inputs,
                        const void* weights, const void* grad_out, void* expz, void* grad_inputs,
                        void* grad_weights, void* ws, size_t ws_bytes, hipStream_t stream) {
    int rc = run(h, dtype, batch, QL_MODE_FWD_BWD, inputs, weights, grad_out, expz, grad_inputs,
                 grad_weights, ws, ws_bytes, stream);
    if (rc == QL_OK) g_err.clear();
    return rc;
}

int ql_forward_backward_static(const ql_circuit* h, ql_dtype dtype, int64_t batch, const void* inputs,
                               const void* weights, const void* grad_out, void* expz, void* grad_inputs,
                               void* grad_weights, hipStream_t stream) {
    if (!h) return fail(QL_EINVAL, "circuit is NULL");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    Layout L;
    int rc = compute_layout(h, (int)dtype, batch, QL_MODE_FWD_BWD, L);
    if (rc) return rc;
    if (L.total > QL_STATIC_SCRATCH_BYTES)
        return fail(QL_ENOMEM, "ql_forward_backward_static needs " + std::to_string(L.total) +
                                   " bytes of scratch, above its static maximum of " +
                                   std::to_string((size_t)QL_STATIC_SCRATCH_BYTES) +
                                   " (use ql_forward_backward with a workspace)");
    void* ws = nullptr;
    if ((rc = static_scratch(&ws))) return rc;
    rc = run(h, dtype, batch, QL_MODE_FWD_BWD, inputs, weights, grad_out, expz, grad_inputs, grad_weights, ws,
             QL_STATIC_SCRATCH_BYTES, stream, true);
    if (rc == QL_OK) g_err.clear();
    return rc;
}

int ql_param_shift_workspace_bytes(const ql_circuit* h, ql_dtype dtype, int64_t batch, int64_t max_chunk,
                                   size_t* out) {
    if (!h || !out) return fail(QL_EINVAL, "NULL argument");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    ShiftLayout S;
    int rc = shift_layout(h, (int)dtype, batch, max_chunk, S);
    if (rc) return rc;
    *out = S.bytes;
    return QL_OK;
}

int ql_param_shift(const ql_circuit* h, ql_dtype dtype, int64_t batch, const void* inputs,
                   const void* weights, const void* grad_out, void* expz, void* grad_inputs,
                   void* grad_weights, int64_t max_chunk, void* ws, size_t ws_bytes, hipStream_t stream) {
    int rc = param_shift(h, dtype, batch, inputs, weights, grad_out, expz, grad_inputs, grad_weights,
                         max_chunk, ws, ws_bytes, stream);
    if (rc == QL_OK) g_err.clear();
    return rc;
}

int ql_state_workspace_bytes(const ql_circuit* h, ql_dtype dtype, int64_t batch, size_t* out) {
    if (!h || !out) return fail(QL_EINVAL, "NULL argument");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    Layout L;
    int rc = compute_layout(h, (int)dtype, batch, QL_MODE_FWD, L, false);
    if (rc) return rc;
    *out = L.total;
    return QL_OK;
}

int ql_state(const ql_circuit* h, ql_dtype dtype, int64_t batch, const void* inputs, const void* weights,
             void* psi, void* ws, size_t ws_bytes, hipStream_t stream) {
    int rc = state(h, dtype, batch, inputs, weights, psi, ws, ws_bytes, stream);
    if (rc == QL_OK) g_err.clear();
    return rc;
}

int ql_sample_workspace_bytes(int32_t n_qubits, int64_t batch, size_t* out) {
    if (!out) return fail(QL_EINVAL, "NULL argument");
    size_t b;
    int rc = sample_bytes(n_qubits, batch, b);
    if (rc) return rc;
    *out = b;
    g_err.clear();
    return QL_OK;
}

int ql_sample(ql_dtype dtype, int32_t n_qubits, int64_t batch, const void* psi, int64_t shots,
              const double* uniforms, int64_t* samples, void* zhat, void* ws, size_t ws_bytes,
              hipStream_t stream) {
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    if (dtype == QL_C128 && n_qubits > QL_MAX_QUBITS_C128) return fail(QL_EUNSUPPORTED, "too many qubits for this dtype");
    size_t need;
    int rc = sample_bytes(n_qubits, batch, need);
    if (rc) return rc;
    if (shots < 0) return fail(QL_EINVAL, "shots must be >= 0");
    if (!psi) return fail(QL_EINVAL, "psi is NULL");
    if (shots > 0 && (!uniforms || !samples)) return fail(QL_EINVAL, "uniforms or samples is NULL");
    if (!ws) return fail(QL_EINVAL, "workspace is NULL");
    if (ws_bytes < need)
        return fail(QL_ENOMEM, "workspace too small: need " + std::to_string(need) + " bytes, got " +
                                   std::to_string(ws_bytes));
    if (batch > ((int64_t)1 << 40) / std::max<int64_t>(shots, 1)) return fail(QL_EINVAL, "batch * shots too large");
    rc = ensure_device();
    if (rc) return rc;
    SampleArgs a{};
    a.psi = psi;
    a.uniforms = uniforms;
    a.samples = samples;
    a.zhat = shots > 0 ? zhat : nullptr;
    a.bsum = (double*)ws;
    a.B = batch;
    a.shots = shots;
    a.n = n_qubits;
    rc = sample_blocks(n_qubits, a.bb, a.nblk);
    if (rc) return rc;
    a.csum = (double*)((char*)ws + align256((size_t)batch * (size_t)a.nblk * 8));
    hipError_t e = launch_sample((int)dtype, a, stream);
    if (e != hipSuccess) return fail(QL_EHIP, std::string("sampling: ") + hipGetErrorString(e));
    g_err.clear();
    return QL_OK;
}

const char* ql_last_error(void) { return g_err.c_str(); }

int ql_plan_info_get(const ql_circuit* h, ql_dtype dtype, ql_plan_info* out) {
    if (!h || !out) return fail(QL_EINVAL, "NULL argument");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    const Plan& pl = h->c.plan[(int)dtype];
    ql_plan_info r{};
    r.kernel = pl.whole_state ? 0 : 1;
    r.n_passes = (int)pl.passes.size();
    r.tile_qubits = pl.k;
    r.log_regs = pl.log_r;
    r.log_threads = pl.log_t;
    r.low_qubits = pl.low;
    for (const auto& pp : pl.passes) {
        r.n_transposes += pp.n_transposes;
        r.n_lane_swaps += pp.n_lane_swaps;
    }
    r.n_rz_groups = (int)pl.diags.size();
    r.n_ryz_pairs = (int)pl.fuses.size();
    r.n_param_gates = h->c.n_param_slots;
    r.n_prefix_gates = (int)pl.pre_gates.size();
    r.n_cz_groups = (int)pl.czgs.size();
    *out = r;
    return QL_OK;
}

int ql_plan_schedule(const ql_circuit* h, ql_dtype dtype, int32_t* pass_of_gate, int32_t* order) {
    if (!h || !pass_of_gate || !order) return fail(QL_EINVAL, "NULL argument");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    const Plan& pl = h->c.plan[(int)dtype];
    // a gate as given is reported at its last piece after intake (a
    // controlled rotation or Pauli channel becomes several gates); gates with
    // no piece (a channel with all probabilities 0) come first, with pass -1
    const int G = h->c.n_user_gates;
    std::vector<int> last(G, -1);
    for (int i = 0; i < G; i++) pass_of_gate[i] = -1;
    int k = 0;
    for (int gi : pl.pre_gates) {  // the product-state prefix: the first pass's initial state
        const int u = h->c.gates[gi].user;
        last[u] = k++;
        pass_of_gate[u] = 0;
    }
    for (int p = 0; p < (int)pl.passes.size(); p++)
        for (int gi : pl.passes[p].gates) {
            const int u = h->c.gates[gi].user;
            last[u] = k++;
            pass_of_gate[u] = p;
        }
    std::vector<std::pair<int, int>> at;
    for (int u = 0; u < G; u++) at.push_back({last[u], u});
    std::sort(at.begin(), at.end());
    for (int i = 0; i < G; i++) order[i] = at[i].second;
    return QL_OK;
}

int ql_plan_state_bytes(const ql_circuit* h, ql_dtype dtype, int64_t batch, int mode, double* out) {
    if (!h || !out) return fail(QL_EINVAL, "NULL argument");
    if (dtype != QL_C64 && dtype != QL_C128) return fail(QL_EINVAL, "unknown dtype");
    const Plan& pl = h->c.plan[(int)dtype];
    const double S = (double)batch * (double)((size_t)1 << h->c.n) * (dtype == QL_C64 ? 8.0 : 16.0);
    const int m = (int)pl.passes.size();
    double units = 0;
    if (!pl.whole_state && m > 1)
        units = mode == QL_MODE_FWD_BWD ? 6.0 * m - 6.0 : mode == QL_MODE_FWD_BWD_KEEP ? 5.0 * m - 5.0 : 2.0 * m - 2.0;
    // with a product prefix the last backward pass also stores lambda
    if (!pl.whole_state && pl.product && (mode == QL_MODE_FWD_BWD || mode == QL_MODE_FWD_BWD_KEEP)) units += 1.0;
    *out = units * S;
    return QL_OK;
}

int ql_timing_enable(ql_circuit* h, int enable) {
    if (!h) return fail(QL_EINVAL, "NULL argument");
    if (enable < 0 || enable > 15) return fail(QL_EINVAL, "timing mask out of range [0, 15]");
    h->timing = enable;
    h->ev_used = 0;
    return QL_OK;
}

int ql_timing_read(ql_circuit* h, double ms[4], int32_t launches[4]) {
    if (!h || !ms || !launches) return fail(QL_EINVAL, "NULL argument");
    for (int i = 0; i < 4; i++) {
        ms[i] = 0;
        launches[i] = 0;
    }
    if (h->ev_used > 0) {
        hipError_t e = hipEventSynchronize(h->ev[h->ev_used - 1].b);
        if (e != hipSuccess) return fail(QL_EHIP, std::string("hipEventSynchronize: ") + hipGetErrorString(e));
    }
    for (size_t i = 0; i < h->ev_used; i++) {
        float t = 0;
        if (hipEventElapsedTime(&t, h->ev[i].a, h->ev[i].b) == hipSuccess) {
            ms[h->ev[i].cls] += t;
            launches[h->ev[i].cls]++;
        }
    }
    h->ev_used = 0;
    return QL_OK;
}

}  // extern "C"
