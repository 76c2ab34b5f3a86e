// Host runtime of the carry-through checksum library: the C ABI declared in
// include/ctc.h.  Builds protected parameters (Sec. II-A, Eq. 1, Sec. II-B),
// folds and packs them for the gfx950 kernels, orders the forward pass on a
// HIP stream, runs the detector and schedules re-execution (Sec. II-B),
// and applies single-bit faults for campaigns (Sec. III-A).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <memory>
#include <string>
#include <vector>

#include "../../include/ctc.h"
#include "kernels.h"

using namespace ctc;

namespace {

thread_local std::string g_err;

ctc_status fail(ctc_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

#define HIP_TRY(expr)                                                        \
    do {                                                                     \
        hipError_t e_ = (expr);                                              \
        if (e_ != hipSuccess)                                                \
            return fail(CTC_ERR_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

constexpr double BN_EPS = 1e-5;
constexpr size_t ALIGN = 256;

size_t align_up(size_t v) { return (v + ALIGN - 1) / ALIGN * ALIGN; }
int round4(int v) { return (v + 3) / 4 * 4; }

uint16_t f32_to_f16_bits(float v) {
    _Float16 h = (_Float16)v;          // round to nearest even
    uint16_t b;
    memcpy(&b, &h, 2);
    return b;
}
// binary16 pattern -> the binary32 pattern of the same value.  Written on
// the integer patterns (no conversion instruction), so it is exact for
// every pattern and a NaN keeps its payload, quiet bit clear or not: a
// stored fp16 weight and its fp32 host copy stay in one-to-one
// correspondence under single-bit faults.
uint32_t f16_widen_bits(uint16_t h) {
    const uint32_t s = (uint32_t)(h >> 15) << 31;
    const int e = (h >> 10) & 31;
    const uint32_t f = h & 1023u;
    if (e == 31) return s | 0x7f800000u | (f << 13);        // Inf, NaN
    if (e > 0) return s | (uint32_t)(e + 112) << 23 | (f << 13);
    if (f == 0) return s;                                   // +-0
    const int sh = __builtin_clz(f) - 21;                   // subnormal:
    return s | (uint32_t)(113 - sh) << 23 | ((f << sh) & 1023u) << 13;
}
uint32_t f32_bits(float v) { uint32_t b; memcpy(&b, &v, 4); return b; }
float bits_f32(uint32_t b) { float v; memcpy(&v, &b, 4); return v; }

struct TensorInfo {
    int c = 0, h = 0, w = 0;   // logical
    int cs = 0;                // stored channels
    int dt = DT_F32;           // storage type
    size_t img_elems = 0, img_bytes = 0;
    size_t off = 0;            // workspace offset (2*max_batch images)
};

struct OpPlan {
    ctc_op spec{};
    int role = CTC_ROLE_NONE;
    int in_has_ck = 0;
    bool dw = false;
    // deployed canonical parameters (construction applied, faults applied)
    std::vector<float> w, b, mean, var, gamma, beta;
    // fp16 nets: the deployed binary16 pattern of every weight in w (w holds
    // its exact fp32 value); single-bit faults XOR these patterns
    std::vector<uint16_t> w16;
    int rows = 0;              // FC: deployed rows
    // workspace offsets
    size_t w_off = 0, w_bytes = 0, sc_off = 0, sh_off = 0;
    int n_out = 0;             // channels / features out (deployed)
    int ktot = 0;              // conv: R*S*Cs_in
    // fusion: 3 on the expand conv of a fusable expand -> depthwise ->
    // project triple (it runs all three), 2 on the first conv of a fusable
    // identity basic block (it runs both convs), 4 on the first conv of a
    // fusable downsampling basic block (conv, shortcut, conv), 5 on a stem
    // conv fusable into the identity block after it (runs all three), 6 on
    // a GAP fusable with the small FC after it, 7 on an fp16 7x7 stride-2
    // stem fusable with the max pool after it, 8 on a dense conv whose
    // output only feeds a 2x2 stride-2 max pool (the pool in its epilogue,
    // where the conv's kernel supports it), 0 else
    int fuse = 0;
    // on a fuse-2 block: the GAP + small FC after it can run in the
    // block's kernel (fuse 6 on the GAP, the block output read only by it)
    bool head = false;
};

struct AppliedFault {
    ctc_fault f;
};

// One queued inference: the staged input in a ring slot and where its
// output row (logits, then S) and flag byte go.
struct Item {
    int slot;
    float *out;                // device address of the output row
    uint8_t *flags;            // device address of the flag byte, or null
    int img;                   // image index in its call (first run), or -1
    bool first;                // first execution (verified) or re-run
    long call = -1;            // forward call that brought it (first runs)
    int old_slot = -1;         // slot it was copied from for this pass: freed
                               // when the pass is settled
};

// A forward pass in flight: tables in pinned host memory, detector event.
struct PassRec {
    RowEnt *rows = nullptr;    // pinned [max_batch]
    StageEnt *stage = nullptr; // pinned [2 * max_batch]
    ActFault *faults = nullptr;// pinned [af_cap], rows resolved
    uint8_t *flagrow = nullptr;// pinned [max_batch]: the detector's flags,
                               // copied from flagdev by the first kernel of
                               // the next pass (or by a flush)
    uint8_t *flagdev = nullptr;// device [max_batch] in the workspace
    hipEvent_t ev = nullptr;   // end of the pass
    hipEvent_t ev_flags = nullptr; // flags copied by a flush
    long no = -1;              // pass number
    long deliver = -1;         // pass whose first kernel copies the flags
                               // (-1: none yet, -2: a flush copied them)
    bool has_ev = false;       // ev recorded after this pass (only some
                               // passes record one: each costs ~2.5 us of
                               // GPU time at the pass boundary)
    bool recorded = false;     // enqueued, not yet settled
    bool harvest = false;      // its flags feed the re-execution queue
    std::vector<Item> items;   // host copy of the rows
};

constexpr int NPASS = 8;       // pass records in rotation
constexpr int SETTLE_LAG = 6;  // a call settles the pass this many back
constexpr int RING_BATCHES = 16;// ring slots = RING_BATCHES * max_batch:
                               // room for a run of max_batch slots per
                               // call with SETTLE_LAG passes unsettled

}  // namespace

struct ctc_net {
    std::vector<OpPlan> ops;
    std::vector<TensorInfo> t;      // tensors 0 .. n_ops-1 (final is caller's)
    int in_c = 0, in_h = 0, in_w = 0, classes = 0, dt = DT_F32, protect = 0;
    int out_cols = 0;
    // append mode: the caller's ops (parameters are given for these) and
    // the widened ops the plan runs
    bool append = false;
    std::vector<ctc_op> user_ops;
    int fusion = CTC_FUSE_IR | CTC_FUSE_BLOCK | CTC_FUSE_STEM | CTC_FUSE_POOL;   // in effect
    // binding
    bool bound = false;
    char *ws = nullptr;
    size_t ws_bytes = 0;
    int max_batch = 0;
    float ref = 0.f, tau = INFINITY;
    // re-execution scheduler
    PassRec pass[NPASS];
    long npass = 0;                 // passes issued
    size_t ring_off = 0, rowsdev_off = 0, cnt_off = 0, flagdev_off = 0;
    // harvested passes whose flags no kernel has copied to host memory
    // yet: a pass's first kernel copies them once FLAG_SEGS wait (a
    // kernel's writes to host memory cost ~5.5 us of the pass they are in,
    // for one flag row as for several)
    std::vector<long> undelivered;
    long last_ev = -1;              // last pass that recorded its event
    size_t part_off = 0, part_bytes = 0;   // split-K partial sums
    int ring_slots = 0;
    std::vector<char> slot_busy;
    int slot_cursor = 0;
    std::deque<Item> queue;         // waiting inferences, FIFO
    long ncall = 0;                 // forward calls in re-executing modes
    // faults
    std::vector<AppliedFault> pfaults;
    // armed activation faults: (tensor id, fault with image = call image)
    std::vector<std::pair<int, ActFault>> afaults;
    std::vector<std::vector<int>> af_by_image;    // indices into afaults
    int af_cap = 0;
    // a pass is being captured into a HIP graph: no flag copies of other
    // passes and no pass events go into it
    bool capture = false;
    // per-stage event timing (measurement support)
    bool prof = false;
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;
    std::vector<std::vector<std::pair<size_t, size_t>>> prof_marks;

    ~ctc_net() {
        for (auto &p : pass) {
            if (p.ev) (void)hipEventDestroy(p.ev);
            if (p.ev_flags) (void)hipEventDestroy(p.ev_flags);
            if (p.rows) (void)hipHostFree(p.rows);
            if (p.stage) (void)hipHostFree(p.stage);
            if (p.faults) (void)hipHostFree(p.faults);
            if (p.flagrow) (void)hipHostFree(p.flagrow);
        }
        for (auto e : ev_pool) (void)hipEventDestroy(e);
    }
};

namespace {

// ------------------------------------------------------- role derivation

// Sec. II-A: every conv gets a carry-through (SUM) filter except the first
// conv of a residual block (ZERO, the add brings the incoming checksum
// back); a depthwise conv and a 1x1 projection shortcut pass the incoming
// checksum through (PASS).
int derive_role(const ctc_op &o) {
    if (o.groups > 1) return CTC_ROLE_PASS;
    if (o.shortcut) return CTC_ROLE_PASS;
    if (o.block_first) return CTC_ROLE_ZERO;
    return CTC_ROLE_SUM;
}

ctc_status build_conv(const ctc_layer_desc *d, float *w, float *bias,
                      float *mean, float *var, float *gamma, float *beta) {
    const int K = d->c_out, C = d->c_in, G = d->groups;
    const int Cg = C / G, R = d->kh, S = d->kw;
    const int r0 = R / 2, s0 = S / 2;
    auto W = [&](int k, int c, int r, int s) -> float & {
        return w[(((size_t)k * Cg + c) * R + r) * S + s];
    };
    if (d->role == CTC_ROLE_NONE) return CTC_OK;
    // input-channel level: normal filters ignore the incoming checksum
    if (d->in_has_ck && G == 1)
        for (int k = 0; k < K - 1; k++)
            for (int r = 0; r < R; r++)
                for (int s = 0; s < S; s++) W(k, C - 1, r, s) = 0.f;
    // output-channel level: replace the last filter
    for (int c = 0; c < Cg; c++)
        for (int r = 0; r < R; r++)
            for (int s = 0; s < S; s++) W(K - 1, c, r, s) = 0.f;
    if (d->role == CTC_ROLE_SUM) {
        for (int c = 0; c < Cg; c++) W(K - 1, c, r0, s0) = 1.f;
    } else if (d->role == CTC_ROLE_PASS) {
        if (G > 1) W(K - 1, 0, r0, s0) = 1.f;
        else if (d->in_has_ck) W(K - 1, C - 1, r0, s0) = 1.f;
    }
    if (bias) bias[K - 1] = 0.f;
    if (mean) {                       // identity entries of Eq. (1)
        mean[K - 1] = 0.f;
        var[K - 1] = 1.f;
        gamma[K - 1] = 1.f;
        beta[K - 1] = 0.f;
    }
    return CTC_OK;
}

ctc_status validate_desc(const ctc_layer_desc *d) {
    if (!d) return fail(CTC_ERR_ARG, "NULL layer descriptor");
    if (d->c_in < 1 || d->c_out < 1 || d->kh < 1 || d->kw < 1 ||
        d->stride < 1 || d->pad < 0 || d->groups < 1)
        return fail(CTC_ERR_ARG, "bad conv sizes");
    if (d->c_in % d->groups || d->c_out % d->groups)
        return fail(CTC_ERR_ARG, "groups must divide c_in and c_out");
    if (d->groups > 1 && !(d->groups == d->c_in && d->c_in == d->c_out))
        return fail(CTC_ERR_UNSUPPORTED, "grouped conv must be depthwise");
    if (d->role < CTC_ROLE_NONE || d->role > CTC_ROLE_PASS)
        return fail(CTC_ERR_ARG, "bad role %d", d->role);
    if (d->role != CTC_ROLE_NONE && (d->kh % 2 == 0 || d->kw % 2 == 0))
        return fail(CTC_ERR_UNSUPPORTED, "carry-through needs odd kernels");
    return CTC_OK;
}

// -------------------------------------------------------------- packing

void fold(const OpPlan &op, std::vector<float> &sc, std::vector<float> &sh) {
    const int n = op.n_out;
    sc.assign(n, 1.f);
    sh.assign(n, 0.f);
    for (int k = 0; k < n; k++) {
        double bias = op.b.empty() ? 0.0 : op.b[k];
        if (!op.mean.empty()) {
            double s = (double)op.gamma[k] / std::sqrt((double)op.var[k] + BN_EPS);
            sc[k] = (float)s;
            sh[k] = (float)((double)op.beta[k] - (double)op.mean[k] * s + bias * s);
        } else {
            sh[k] = (float)bias;
        }
    }
}

// FC weights are stored fragment-major, so that one wave's weights for one
// k step (16 output rows x KS k, the MFMA A fragment) are 1 KB of
// contiguous memory: fragment [row / 16][k / KS], inside it lane
// (k % KS) / KG * 16 + row % 16 holds KG consecutive k.  KS, KG = 32, 8
// for fp16 weights, 16, 4 for fp32 ones.  Layers past fc_small store the
// fragments of 64-row blocks together: [row / 64][k / KS][row / 16 % 4].
// Rows past the layer's (to 16, or 64) and k past its inputs are zero.
void fc_frag(const ctc_net *net, const OpPlan &, int *ks, int *kg) {
    const bool w16 = net->dt == DT_F16;
    *ks = w16 ? 32 : 16;
    *kg = w16 ? 8 : 4;
}

// Physical element index of deployed canonical weight element `idx`.
size_t packed_index(const ctc_net *net, const OpPlan &op, size_t idx) {
    const ctc_op &o = op.spec;
    if (o.kind == CTC_OP_CONV) {
        const int R = o.k, S = o.k;
        if (op.dw) {                 // [K][1][R][S] -> [R][S][K]
            size_t rs = idx % (size_t)(R * S), k = idx / (size_t)(R * S);
            return rs * o.c_out + k;
        }
        const int Cg = o.c_in;
        const int Cs = net->t[o.input].cs;
        size_t s = idx % S, r = (idx / S) % R, c = (idx / (S * R)) % Cg,
               k = idx / ((size_t)S * R * Cg);
        return k * op.ktot + (r * S + s) * Cs + c;
    }
    // FC [rows][I]; flatten: canonical c*HW + hw -> device hw*C + c;
    // then the fragment-major order
    const size_t I = o.c_in;
    size_t row = idx / I, i = idx % I;
    if (o.flatten_c > 0) {
        size_t HW = (size_t)o.flatten_h * o.flatten_w;
        size_t c = i / HW, hw = i % HW;
        i = hw * o.flatten_c + c;
    }
    int ks, kg;
    fc_frag(net, op, &ks, &kg);
    const size_t nsteps = (I + ks - 1) / ks, st = i / ks, r = i % ks;
    const size_t ln = (r / kg) * 16 + row % 16;
    if (!fc_small_shape(op.rows, (int)I))
        return ((((row / 64) * nsteps + st) * 4 + (row / 16) % 4) * 64 + ln) * kg + r % kg;
    return (((row / 16) * nsteps + st) * 64 + ln) * kg + r % kg;
}

size_t weight_elems(const ctc_net *net, const OpPlan &op) {
    const ctc_op &o = op.spec;
    if (o.kind == CTC_OP_CONV)
        return op.dw ? (size_t)o.k * o.k * o.c_out : (size_t)o.c_out * op.ktot;
    int ks, kg;
    fc_frag(net, op, &ks, &kg);
    const int rb = fc_small_shape(op.rows, o.c_in) ? 16 : 64;
    return (size_t)(op.rows + rb - 1) / rb * rb * ((o.c_in + ks - 1) / ks) * ks;
}

int wbytes(const ctc_net *net) { return net->dt == DT_F16 ? 2 : 4; }

void pack_weights(const ctc_net *net, const OpPlan &op, std::vector<char> &buf) {
    const size_t n = weight_elems(net, op);
    const int eb = wbytes(net);
    buf.assign(n * eb, 0);
    for (size_t i = 0; i < op.w.size(); i++) {
        size_t p = packed_index(net, op, i);
        if (eb == 4) memcpy(&buf[p * 4], &op.w[i], 4);
        else {
            const uint16_t h = op.w16.size() == op.w.size() ? op.w16[i]
                                                            : f32_to_f16_bits(op.w[i]);
            memcpy(&buf[p * 2], &h, 2);
        }
    }
}

// ------------------------------------------------------------ forward pass

hipStream_t S(void *s) { return (hipStream_t)s; }

// Dense conv: spatial-tile kernel where it applies, else implicit GEMM.
hipError_t launch_any_conv(int dt, const ConvArgs &a, hipStream_t st) {
    if (a.pool) return launch_conv(dt, a, st);       // pooled: implicit GEMM only
    TileCfg tc = choose_tile(dt, a);
    if (tc.IMW > 0) return launch_conv_tile(dt, a, tc, st);
    return launch_conv(dt, a, st);
}

// Whether the fusable basic block starting at op i runs fused for a pass of
// nimg images: only when its tiles fill the GPU at least once (below that,
// the two separate convs spread over more workgroups and finish sooner).
bool block_fused(const ctc_net *net, int i, int nimg) {
    const TensorInfo &tx = net->t[net->ops[i].spec.input];
    // the 64-channel block's 4x8 tiles recompute conv1 on a 6x10 region:
    // 1.25x the work on an 8x8 map, nearly 2x on larger ones (ResNet-18's
    // 56x56 stage ran 351 us fused against ~296 us as two convs)
    if (tx.cs == 64 && (tx.h > 8 || tx.w > 8)) return false;
    BlockArgs b{};
    b.nimg = nimg; b.H = tx.h; b.W = tx.w; b.C = tx.cs;
    choose_block_tile(b);
    if (b.TH == 0) return false;
    const long tiles = (long)nimg * ((b.W + b.TW - 1) / b.TW) * ((b.H + b.TH - 1) / b.TH);
    return tiles >= 256;
}

// When profiling, arms two pool events for the next kernel launch (they
// receive the kernel's own start / end timestamps); returns the index of
// the first or -1.
long prof_mark(ctc_net *net, hipStream_t) {
    if (!net->prof) return -1;
    while (net->ev_used + 2 > net->ev_pool.size()) {
        hipEvent_t e;
        // timing only: without the system-scope fence the event does not
        // write back and invalidate L2 at the kernel's end, which would add
        // that cost to the measured launch and to the next one
        if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess)
            return -1;
        net->ev_pool.push_back(e);
    }
    size_t i = net->ev_used;
    net->ev_used += 2;
    set_launch_events(net->ev_pool[i], net->ev_pool[i + 1]);
    return (long)i;
}

void prof_close(ctc_net *net, int slot, long begin, hipStream_t) {
    if (begin < 0) return;
    if (launch_events_pending()) {      // nothing was launched
        set_launch_events(nullptr, nullptr);
        net->ev_used -= 2;
        return;
    }
    net->prof_marks[slot].push_back({(size_t)begin, (size_t)begin + 1});
}

// Runs one pass over the rows in `p` (their tables already written):
// input assembly, every layer, detector.  x: the caller's batch for work
// items that convert fresh images (may be null).
ctc_status run_pass(ctc_net *net, PassRec &p, int nstage, const float *x,
                    hipStream_t st, char *in0 = nullptr) {
    const int nr = (int)p.items.size();
    char *ws = net->ws;
    const TensorInfo &t0 = net->t[0];
    // the pass's input rows: tensor 0's buffer, or a run of ring slots
    const bool in_ring = in0 != nullptr;
    if (!in_ring) in0 = ws + t0.off;
    auto tp = [&](int t) -> char * { return t == 0 ? in0 : ws + net->t[t].off; };
    RowEnt *rows_dev = (RowEnt *)(ws + net->rowsdev_off);
    // armed activation faults, resolved to the rows of first executions
    const int ntens = (int)net->ops.size() + 1;
    std::vector<std::vector<ActFault>> res(ntens);
    int nf = 0;
    if (!net->afaults.empty()) {
        for (int r = 0; r < nr; r++) {
            const Item &it = p.items[r];
            if (!it.first || it.img < 0 || it.img >= (int)net->af_by_image.size())
                continue;
            for (int k : net->af_by_image[it.img]) {
                // several calls' rows may share an image index: refuse
                // rather than drop faults past the pinned table
                if (nf >= net->af_cap)
                    return fail(CTC_ERR_STATE,
                                "more than %d armed activation faults in one pass",
                                net->af_cap);
                ActFault g = net->afaults[k].second;
                g.image = r;
                res[net->afaults[k].first].push_back(g);
                nf++;
            }
        }
    }
    std::vector<int> per_t(ntens, 0), first_t(ntens, 0);
    for (int t = 0, o = 0; t < ntens; t++) {
        first_t[t] = o;
        per_t[t] = (int)res[t].size();
        for (const ActFault &g : res[t]) p.faults[o++] = g;
    }
    auto apply_act = [&](int tid, void *base, size_t img_bytes) -> ctc_status {
        if (per_t[tid] > 0)
            HIP_TRY(launch_act_faults(base, img_bytes, p.faults + first_t[tid],
                                      per_t[tid], nr, st));
        return CTC_OK;
    };
    // a fault on the input would reach the copy that a re-execution reads
    if (in_ring && per_t[0] > 0)
        return fail(CTC_ERR_STATE, "input fault on a pass that reads the ring");
    const int nops = (int)net->ops.size();
    // whether op i and the two after it run as one fused stem + block kernel
    auto stem_block = [&](int i) {
        return i + 2 < nops && net->ops[i].fuse == 5 && (net->fusion & CTC_FUSE_BLOCK) &&
               per_t[i + 1] == 0 && per_t[i + 2] == 0 && block_fused(net, i + 1, nr);
    };
    // When the pass's first kernel is a fused stem + block, that kernel
    // stages the input itself (and copies the row table): no separate
    // assembly launch.  It takes the usual shape of a pass: rows 0..n-1
    // converted from the caller's images 0..n-1, then up to BLOCK_STAGE_MAX
    // rows from ring slots (re-executions), plus up to BLOCK_STAGE_MAX more
    // of the caller's images converted into ring slots for later passes.
    BlockArgs stage{};
    bool direct = x && nr > 0 && per_t[0] == 0 && stem_block(0) && t0.dt == DT_F32 &&
                  t0.cs == 4 && net->in_c >= 1 && net->in_c <= 4 && (uintptr_t)x % 4 == 0;
    {
        int nrr = 0, maxsrc = -1;
        for (int k = 0; direct && k < nstage; k++) {
            const StageEnt &g = p.stage[k];
            if (g.src >= 0 && g.slot < 0 && g.row == g.src && g.row == stage.xs_n && nrr == 0) {
                stage.xs_n++;
            } else if (g.src < 0 && g.slot >= 0 && g.row == stage.xs_n + nrr &&
                       nrr < BLOCK_STAGE_MAX) {
                stage.rr_slot[nrr++] = g.slot;
            } else if (g.src >= 0 && g.slot >= 0 && g.row < 0 &&
                       stage.ov_n < BLOCK_STAGE_MAX) {
                stage.ov_src[stage.ov_n] = g.src;
                stage.ov_slot[stage.ov_n++] = g.slot;
            } else {
                direct = false;
            }
            if (g.src > maxsrc) maxsrc = g.src;
        }
        direct = direct && stage.xs_n + nrr == nr;
        stage.xs = x;
        stage.xs_c = net->in_c;
        stage.xs_imgs = maxsrc + 1;
        stage.ring = ws + net->ring_off;
        stage.ring_bytes = (long)RING_BATCHES * net->max_batch * t0.img_bytes;
        stage.rows_host = p.rows;
        stage.rows_dev = rows_dev;
        stage.nrows = nr;
        if (direct) {                    // sizes the kernel accepts
            BlockArgs chk = stage;
            const TensorInfo &tb = net->t[1];
            chk.nimg = nr; chk.H = tb.h; chk.W = tb.w; chk.C = tb.cs;
            chk.x0 = in0;
            choose_block_tile(chk);
            direct = block_ok(chk);
        }
    }
    // the flags of the harvested pass before this one go to host memory in
    // this pass's first kernel (early in it, not at a pass's end)
    FlagCopy fcopy{};
    std::vector<PassRec *> fpass;
    if (!net->capture && (int)net->undelivered.size() >= FLAG_SEGS) {
        for (long no : net->undelivered) {
            PassRec &m = net->pass[no % NPASS];
            if (fcopy.nseg < FLAG_SEGS && m.no == no && m.recorded && m.harvest &&
                m.deliver < 0) {
                fcopy.src[fcopy.nseg] = m.flagdev;
                fcopy.dst[fcopy.nseg] = m.flagrow;
                fcopy.n[fcopy.nseg++] = (int)m.items.size();
                fpass.push_back(&m);
            }
        }
    }
    auto delivered = [&]() {
        for (PassRec *m : fpass) {
            m->deliver = p.no;
            auto &u = net->undelivered;
            u.erase(std::remove(u.begin(), u.end(), m->no), u.end());
        }
        fpass.clear();
    };
    long pm;
    if (!direct) {
        pm = prof_mark(net, st);
        HIP_TRY(launch_assemble(t0.dt, x, net->in_c, net->in_h, net->in_w, t0.cs,
                                p.stage, nstage, ws + net->ring_off, in0,
                                p.rows, rows_dev, nr, fcopy, st));
        prof_close(net, 0, pm, st);
        delivered();
    }
    ctc_status s = apply_act(0, in0, t0.img_bytes);
    if (s != CTC_OK) return s;
    // arguments of FC op j on input x; *dout = its output type
    auto fc_args = [&](int j, const void *x, int *dout) {
        const OpPlan &fo = net->ops[j];
        FcArgs a{};
        a.det_col = -1;
        a.x = x;
        a.w = ws + fo.w_off;
        a.shift = (const float *)(ws + fo.sh_off);
        a.nimg = nr;
        a.I = fo.spec.c_in;
        a.O = fo.rows;
        a.relu = fo.spec.relu;
        a.part = net->part_bytes ? (float *)(ws + net->part_off) : nullptr;
        if (j == nops - 1) {
            a.rows = rows_dev;
            *dout = DT_F32;
            // the detector runs in the FC epilogue unless a fault on the
            // stored output must land before it
            a.det_col = (net->protect && per_t[nops] == 0) ? net->classes : -1;
            a.ref = net->ref;
            a.tau = net->tau;
            a.flag_pass = p.flagdev;
        } else {
            const TensorInfo &to = net->t[j + 1];
            a.y = ws + to.off; a.ld = to.cs;
            *dout = to.dt;
        }
        return a;
    };
    for (int i = 0; i < nops; i++) {
        const OpPlan &op = net->ops[i];
        const ctc_op &o = op.spec;
        const TensorInfo &ti = net->t[o.input];
        const bool last = i == nops - 1;
        pm = prof_mark(net, st);
        // a fused block, unless a fault is armed on one of its internal
        // tensors (then the three ops run separately and store them)
        // the stem fused into the identity block after it (when that block
        // runs fused in this pass and the stem output and the block's
        // internal tensor are fault-free)
        // the stem and the max pool after it (stem output fault-free)
        if (op.fuse == 7 && (net->fusion & CTC_FUSE_STEM) && per_t[i + 1] == 0) {
            const TensorInfo &ts = net->t[i + 1], &tq = net->t[i + 2];
            ConvArgs a{};
            a.x = tp(o.input);
            a.w = ws + op.w_off;
            a.scale = (const float *)(ws + op.sc_off);
            a.shift = (const float *)(ws + op.sh_off);
            a.y = ws + tq.off;
            a.nimg = nr;
            a.H = ti.h; a.W = ti.w; a.Cs = ti.cs;
            a.P = ts.h; a.Q = ts.w; a.N = o.c_out;
            a.R = o.k; a.S = o.k; a.stride = o.stride; a.pad = o.pad;
            a.relu = o.relu;
            hipError_t e = launch_stem_pool(a, tq.h, tq.w, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused stem + pool %d: %s", i, hipGetErrorString(e));
            prof_close(net, 1 + i, pm, st);
            i += 1;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        if (stem_block(i)) {
            const OpPlan &b1 = net->ops[i + 1], &b2 = net->ops[i + 2];
            const TensorInfo &tb = net->t[i + 1];
            BlockArgs b{};
            b.x = tp(i + 1);                    // not read with the stem
            b.w1 = ws + b1.w_off;
            b.sc1 = (const float *)(ws + b1.sc_off);
            b.sh1 = (const float *)(ws + b1.sh_off);
            b.w2 = ws + b2.w_off;
            b.sc2 = (const float *)(ws + b2.sc_off);
            b.sh2 = (const float *)(ws + b2.sh_off);
            b.y = ws + net->t[i + 3].off;
            b.nimg = nr; b.H = tb.h; b.W = tb.w; b.C = tb.cs;
            b.x0 = tp(o.input);
            b.w0 = ws + op.w_off;
            b.sc0 = (const float *)(ws + op.sc_off);
            b.sh0 = (const float *)(ws + op.sh_off);
            if (direct && i == 0) {
                b.xs = stage.xs; b.xs_c = stage.xs_c;
                b.xs_n = stage.xs_n; b.xs_imgs = stage.xs_imgs;
                b.ring = stage.ring; b.ring_bytes = stage.ring_bytes;
                std::copy(stage.rr_slot, stage.rr_slot + BLOCK_STAGE_MAX, b.rr_slot);
                b.ov_n = stage.ov_n;
                std::copy(stage.ov_src, stage.ov_src + BLOCK_STAGE_MAX, b.ov_src);
                std::copy(stage.ov_slot, stage.ov_slot + BLOCK_STAGE_MAX, b.ov_slot);
                b.rows_host = stage.rows_host; b.rows_dev = stage.rows_dev;
                b.nrows = stage.nrows;
                b.flags = fcopy;
            }
            choose_block_tile(b);
            hipError_t e = launch_block(b, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused stem + block %d: %s", i, hipGetErrorString(e));
            if (direct && i == 0) delivered();
            prof_close(net, 1 + i, pm, st);
            i += 2;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        // a fused downsampling block (its two internal tensors fault-free)
        if (op.fuse == 4 && (net->fusion & CTC_FUSE_BLOCK) && per_t[i + 1] == 0 &&
            per_t[i + 2] == 0) {
            const OpPlan &sc = net->ops[i + 1], &o2 = net->ops[i + 2];
            const TensorInfo &to = net->t[i + 3];
            DownArgs d{};
            d.x = tp(o.input);
            d.w1 = ws + op.w_off;
            d.sc1 = (const float *)(ws + op.sc_off);
            d.sh1 = (const float *)(ws + op.sh_off);
            d.ws = ws + sc.w_off;
            d.scs = (const float *)(ws + sc.sc_off);
            d.shs = (const float *)(ws + sc.sh_off);
            d.w2 = ws + o2.w_off;
            d.sc2 = (const float *)(ws + o2.sc_off);
            d.sh2 = (const float *)(ws + o2.sh_off);
            d.y = ws + to.off;
            d.nimg = nr; d.H = ti.h; d.W = ti.w; d.P = to.h; d.Q = to.w;
            d.Ci = ti.cs; d.Co = o.c_out;
            hipError_t e = launch_down(d, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused block %d: %s", i, hipGetErrorString(e));
            prof_close(net, 1 + i, pm, st);
            i += 2;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        // a fused basic block: same rule for its internal tensor
        if (op.fuse == 2 && (net->fusion & CTC_FUSE_BLOCK) && per_t[i + 1] == 0 &&
            block_fused(net, i, nr)) {
            const OpPlan &o2 = net->ops[i + 1];
            BlockArgs b{};
            b.x = tp(o.input);
            b.w1 = ws + op.w_off;
            b.sc1 = (const float *)(ws + op.sc_off);
            b.sh1 = (const float *)(ws + op.sh_off);
            b.w2 = ws + o2.w_off;
            b.sc2 = (const float *)(ws + o2.sc_off);
            b.sh2 = (const float *)(ws + o2.sh_off);
            b.y = ws + net->t[i + 2].off;
            b.nimg = nr; b.H = ti.h; b.W = ti.w; b.C = ti.cs;
            // the GAP + FC behind it in the same kernel (the block output
            // and the pooled tensor fault-free)
            const bool head = op.head && per_t[i + 2] == 0 && per_t[i + 3] == 0;
            if (head) {
                int dout;
                b.fc = fc_args(i + 3, nullptr, &dout);
                b.head = true;
                b.cnt = (int *)(ws + net->cnt_off);
            }
            choose_block_tile(b);
            hipError_t e = launch_block(b, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused block %d: %s", i, hipGetErrorString(e));
            prof_close(net, 1 + i, pm, st);
            i += head ? 3 : 1;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        if (op.fuse == 3 && (net->fusion & CTC_FUSE_IR) && per_t[i + 1] == 0 &&
            per_t[i + 2] == 0) {
            const OpPlan &d = net->ops[i + 1], &pj = net->ops[i + 2];
            const TensorInfo &to = net->t[i + 3];
            IrArgs a{};
            a.x = tp(o.input);
            a.we = ws + op.w_off;
            a.sce = (const float *)(ws + op.sc_off);
            a.she = (const float *)(ws + op.sh_off);
            a.wd = ws + d.w_off;
            a.scd = (const float *)(ws + d.sc_off);
            a.shd = (const float *)(ws + d.sh_off);
            a.wp = ws + pj.w_off;
            a.scp = (const float *)(ws + pj.sc_off);
            a.shp = (const float *)(ws + pj.sh_off);
            a.res = pj.spec.residual >= 0 ? tp(pj.spec.residual) : nullptr;
            a.y = ws + to.off;
            a.nimg = nr;
            a.H = ti.h; a.W = ti.w; a.C = ti.cs; a.E = o.c_out;
            a.Co = pj.spec.c_out; a.P = to.h; a.Q = to.w;
            a.stride = d.spec.stride; a.relu_p = pj.spec.relu;
            hipError_t e = launch_ir(a, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused block %d: %s", i, hipGetErrorString(e));
            prof_close(net, 1 + i, pm, st);
            i += 2;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        // a fused depthwise + pointwise pair (its depthwise output fault-free)
        if (op.fuse == 9 && (net->fusion & CTC_FUSE_IR) && per_t[i + 1] == 0) {
            const OpPlan &pj = net->ops[i + 1];
            DwPwArgs a{};
            a.x = tp(o.input);
            a.wd = ws + op.w_off;
            a.scd = (const float *)(ws + op.sc_off);
            a.shd = (const float *)(ws + op.sh_off);
            a.relu_d = o.relu;
            a.wp = ws + pj.w_off;
            a.scp = (const float *)(ws + pj.sc_off);
            a.shp = (const float *)(ws + pj.sh_off);
            a.res = pj.spec.residual >= 0 ? tp(pj.spec.residual) : nullptr;
            a.y = ws + net->t[i + 2].off;
            a.relu_p = pj.spec.relu;
            a.nimg = nr; a.H = ti.h; a.W = ti.w; a.C = ti.cs; a.Co = pj.spec.c_out;
            hipError_t e = launch_dwpw(a, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused pair %d: %s", i, hipGetErrorString(e));
            prof_close(net, 1 + i, pm, st);
            i += 1;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        // GAP and the small FC after it in one kernel (pooled tensor
        // fault-free)
        if (op.fuse == 6 && (net->fusion & CTC_FUSE_BLOCK) && per_t[i + 1] == 0) {
            int dout;
            FcArgs a = fc_args(i + 1, tp(o.input), &dout);
            hipError_t e = launch_gap_fc(a, ti.h * ti.w, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "fused GAP + FC %d: %s", i, hipGetErrorString(e));
            prof_close(net, 1 + i, pm, st);
            i += 1;
            if (i < nops - 1) {
                s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                if (s != CTC_OK) return s;
            }
            continue;
        }
        // the conv and the 2x2 max pool after it in one kernel (conv output
        // fault-free, a kernel with the pool for this shape)
        if (op.fuse == 8 && (net->fusion & CTC_FUSE_POOL) && per_t[i + 1] == 0) {
            const TensorInfo &to = net->t[i + 1], &tq = net->t[i + 2];
            ConvArgs a{};
            a.x = tp(o.input);
            a.w = ws + op.w_off;
            a.scale = (const float *)(ws + op.sc_off);
            a.shift = (const float *)(ws + op.sh_off);
            a.res = o.residual >= 0 ? tp(o.residual) : nullptr;
            a.y = ws + tq.off;
            a.nimg = nr;
            a.H = ti.h; a.W = ti.w; a.Cs = ti.cs;
            a.P = to.h; a.Q = to.w; a.N = o.c_out;
            a.R = o.k; a.S = o.k; a.stride = o.stride; a.pad = o.pad;
            a.relu = o.relu;
            a.pool = 2;
            if (conv_pool_ok(to.dt, a)) {
                hipError_t e = launch_conv(to.dt, a, st);
                if (e != hipSuccess)
                    return fail(CTC_ERR_DEVICE, "conv + pool %d: %s", i, hipGetErrorString(e));
                prof_close(net, 1 + i, pm, st);
                i += 1;
                if (i < nops - 1) {
                    s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
                    if (s != CTC_OK) return s;
                }
                continue;
            }
        }
        if (o.kind == CTC_OP_CONV) {
            const TensorInfo &to = net->t[i + 1];
            ConvArgs a{};
            a.x = tp(o.input);
            a.w = ws + op.w_off;
            a.scale = (const float *)(ws + op.sc_off);
            a.shift = (const float *)(ws + op.sh_off);
            a.res = o.residual >= 0 ? tp(o.residual) : nullptr;
            a.y = ws + to.off;
            a.nimg = nr;
            a.H = ti.h; a.W = ti.w; a.Cs = ti.cs;
            a.P = to.h; a.Q = to.w; a.N = o.c_out;
            a.R = o.k; a.S = o.k; a.stride = o.stride; a.pad = o.pad;
            a.relu = o.relu;
            a.part = net->part_bytes ? (float *)(ws + net->part_off) : nullptr;
            hipError_t e = op.dw ? launch_dwconv(to.dt, a, st)
                                 : launch_any_conv(to.dt, a, st);
            if (e != hipSuccess)
                return fail(CTC_ERR_DEVICE, "conv %d: %s", i, hipGetErrorString(e));
        } else if (o.kind == CTC_OP_MAXPOOL) {
            const TensorInfo &to = net->t[i + 1];
            HIP_TRY(launch_maxpool(to.dt, tp(o.input), ws + to.off, nr, ti.h,
                                   ti.w, ti.cs, to.h, to.w, o.k, o.stride,
                                   o.pad, st));
        } else if (o.kind == CTC_OP_GAP) {
            const TensorInfo &to = net->t[i + 1];
            HIP_TRY(launch_gap(to.dt, tp(o.input), ws + to.off, nr,
                               ti.h * ti.w, ti.cs, st));
        } else {
            int dout;
            FcArgs a = fc_args(i, tp(o.input), &dout);
            HIP_TRY(launch_fc(ti.dt, net->dt, dout, a, st));
        }
        prof_close(net, 1 + i, pm, st);
        if (!last) {
            s = apply_act(i + 1, ws + net->t[i + 1].off, net->t[i + 1].img_bytes);
            if (s != CTC_OK) return s;
        }
    }
    // faults on the final output (logits || S): row addresses vary, so
    // each is applied through the row table copy on the host side
    for (int k = 0; k < per_t[nops]; k++) {
        const ActFault &f = p.faults[first_t[nops] + k];   // image = pass row
        char *row = (char *)p.items[f.image].out;
        HIP_TRY(launch_act_faults(row, 0, &p.faults[first_t[nops] + k], 1,
                                  f.image + 1, st));
    }
    if (net->protect && per_t[nops] > 0) {
        pm = prof_mark(net, st);
        HIP_TRY(launch_verify_pass(rows_dev, nr, net->classes, net->ref,
                                   net->tau, p.flagdev, st));
        prof_close(net, nops + 1, pm, st);
    }
    // an event ends the passes that copy flags to the host, and any pass
    // FLAG_SEGS after the last one with an event (what waits for a pass
    // uses the first event at or after it)
    if (!net->capture && (fcopy.nseg > 0 || p.no - net->last_ev >= FLAG_SEGS)) {
        HIP_TRY(hipEventRecord(p.ev, st));
        p.has_ev = true;
        net->last_ev = p.no;
    }
    p.recorded = true;
    if (p.harvest) net->undelivered.push_back(p.no);
    return CTC_OK;
}

// Waits for pass record k (if in flight); when it feeds the queue, pushes
// its flagged first executions to the queue front and frees the ring slots
// it no longer needs.  Its flags reach host memory through the first
// kernel of the pass after it (whose end is then waited for) or, when no
// pass has followed yet, through a copy enqueued here on st.
ctc_status settle(ctc_net *net, int k, hipStream_t st) {
    PassRec &p = net->pass[k];
    if (!p.recorded) return CTC_OK;
    if (p.harvest && p.deliver == -2) {
        // copied by a flush, which waited for the copy after the pass
    } else if (p.harvest && p.deliver < 0) {
        // no pass has copied its flags yet: copied here, after it in
        // stream order
        HIP_TRY(hipMemcpyAsync(p.flagrow, p.flagdev, p.items.size(),
                               hipMemcpyDeviceToHost, st));
        HIP_TRY(hipEventRecord(p.ev_flags, st));
        HIP_TRY(hipEventSynchronize(p.ev_flags));
        auto &u = net->undelivered;
        u.erase(std::remove(u.begin(), u.end(), p.no), u.end());
    } else {
        // the end of this pass (and of the one that copied its flags): the
        // first later pass with an event (records of passes after this one
        // are not reused before it is settled), else one recorded now
        PassRec *w = nullptr;
        for (long j = p.harvest ? p.deliver : p.no; j < net->npass && !w; j++) {
            PassRec &q = net->pass[j % NPASS];
            if (q.no == j && q.has_ev) w = &q;
        }
        if (!w) {
            HIP_TRY(hipEventRecord(p.ev, st));
            p.has_ev = true;
            w = &p;
        }
        HIP_TRY(hipEventSynchronize(w->ev));
    }
    p.recorded = false;
    if (!p.harvest) return CTC_OK;
    p.harvest = false;
    // re-runs go to the front, in row order
    for (int r = (int)p.items.size() - 1; r >= 0; r--) {
        const Item &it = p.items[r];
        if (it.old_slot >= 0) net->slot_busy[it.old_slot] = 0;
        if (it.first && p.flagrow[r]) {
            net->queue.push_front(Item{it.slot, it.out, nullptr, -1, false, -1});
        } else if (it.slot >= 0) {
            net->slot_busy[it.slot] = 0;
        }
    }
    return CTC_OK;
}

// Next pass record, waiting for its previous use to finish.
ctc_status next_pass(ctc_net *net, PassRec **out, hipStream_t st) {
    const int k = (int)(net->npass % NPASS);
    ctc_status s = settle(net, k, st);
    if (s != CTC_OK) return s;
    net->pass[k].no = net->npass;
    net->pass[k].deliver = -1;
    net->pass[k].has_ev = false;
    net->npass++;
    net->pass[k].items.clear();
    *out = &net->pass[k];
    return CTC_OK;
}

// Settles every pass record, oldest first.  The flag rows no pass has
// copied yet are copied first, all behind one event.
ctc_status settle_all(ctc_net *net, hipStream_t st) {
    if (!net->undelivered.empty()) {
        PassRec *last = nullptr;
        for (long no : net->undelivered) {
            PassRec &m = net->pass[no % NPASS];
            if (m.no != no || !m.recorded || !m.harvest || m.deliver >= 0) continue;
            HIP_TRY(hipMemcpyAsync(m.flagrow, m.flagdev, m.items.size(),
                                   hipMemcpyDeviceToHost, st));
            m.deliver = net->npass;          // "after every pass issued so far"
            last = &m;
        }
        net->undelivered.clear();
        if (last) {
            HIP_TRY(hipEventRecord(last->ev_flags, st));
            HIP_TRY(hipEventSynchronize(last->ev_flags));
            for (long c = std::max(0l, net->npass - NPASS); c < net->npass; c++) {
                PassRec &m = net->pass[c % NPASS];
                if (m.recorded && m.deliver == net->npass) m.deliver = -2;
            }
        }
    }
    for (long c = net->npass - NPASS; c < net->npass; c++) {
        if (c < 0) continue;
        ctc_status s = settle(net, (int)(c % NPASS), st);
        if (s != CTC_OK) return s;
    }
    return CTC_OK;
}

// Takes up to n items from the queue front into a pass (all from the ring).
ctc_status run_queue_pass(ctc_net *net, int n, hipStream_t st) {
    PassRec *p;
    ctc_status s = next_pass(net, &p, st);
    if (s != CTC_OK) return s;
    int ns = 0;
    for (int r = 0; r < n && !net->queue.empty(); r++) {
        Item it = net->queue.front();
        net->queue.pop_front();
        p->items.push_back(it);
        p->rows[r] = RowEnt{(int64_t)(uintptr_t)it.out,
                            (int64_t)(uintptr_t)it.flags, it.slot, it.first};
        p->stage[ns++] = StageEnt{-1, it.slot, r, 0};
    }
    p->harvest = true;
    return run_pass(net, *p, ns, nullptr, st);
}

int alloc_slot(ctc_net *net) {
    for (int k = 0; k < net->ring_slots; k++) {
        const int c = (net->slot_cursor + k) % net->ring_slots;
        if (!net->slot_busy[c]) {
            net->slot_busy[c] = 1;
            net->slot_cursor = (c + 1) % net->ring_slots;
            return c;
        }
    }
    return -1;
}

// First run of n consecutive free slots from the cursor on (a run does not
// wrap round the ring's end): marks it busy and returns its first slot, or
// -1 when there is none.
int alloc_run(ctc_net *net, int n) {
    const int R = net->ring_slots;
    if (n <= 0 || n > R) return -1;
    int c = net->slot_cursor;
    for (int seen = 0; seen < 2 * R;) {
        if (c + n > R) {
            seen += R - c;
            c = 0;
            continue;
        }
        int k = 0;
        while (k < n && !net->slot_busy[c + k]) k++;
        if (k == n) {
            for (int j = 0; j < n; j++) net->slot_busy[c + j] = 1;
            net->slot_cursor = (c + n) % R;
            return c;
        }
        seen += k + 1;
        c += k + 1;
    }
    return -1;
}

// Whether an activation fault is armed on the network input (tensor 0).
bool input_faults_armed(const ctc_net *net) {
    for (const auto &f : net->afaults)
        if (f.first == 0) return true;
    return false;
}

}  // namespace

// =====================================================================
// C ABI
// =====================================================================
extern "C" {

int32_t ctc_abi_version(void) { return CTC_ABI_VERSION; }
const char *ctc_last_error(void) { return g_err.c_str(); }

ctc_status ctc_build_filters(const ctc_layer_desc *d, float *w, float *bias,
                             float *mean, float *var, float *gamma,
                             float *beta) {
    ctc_status s = validate_desc(d);
    if (s != CTC_OK) return s;
    if (!w) return fail(CTC_ERR_ARG, "NULL weights");
    const bool any_bn = mean || var || gamma || beta;
    if (any_bn && !(mean && var && gamma && beta))
        return fail(CTC_ERR_ARG, "BN needs all of mean, var, gamma, beta");
    return build_conv(d, w, bias, mean, var, gamma, beta);
}

ctc_status ctc_build_fc(int32_t in_f, int32_t out_f, int32_t ck_first,
                        int32_t ck_count, int32_t is_final, const float *w_in,
                        const float *b_in, float *w_out, float *b_out) {
    if (in_f < 1 || out_f < 1 || !w_in || !w_out)
        return fail(CTC_ERR_ARG, "bad FC arguments");
    if (ck_count < 0 || ck_first < 0 || ck_first + ck_count > in_f)
        return fail(CTC_ERR_ARG, "checksum features out of range");
    if (b_in && !b_out) return fail(CTC_ERR_ARG, "b_out needed with b_in");
    if (w_in == w_out) return fail(CTC_ERR_ARG, "w_out aliases w_in");
    const size_t I = in_f;
    const int rows = out_f + (is_final ? 1 : 0);
    const int normal = is_final ? out_f : out_f - 1;
    for (int o = 0; o < rows; o++) {
        float *dst = w_out + o * I;
        if (o < normal) {
            memcpy(dst, w_in + o * I, I * sizeof(float));
            for (int c = ck_first; c < ck_first + ck_count; c++) dst[c] = 0.f;
        } else {
            for (size_t i = 0; i < I; i++) dst[i] = 1.f;  // sums every input
        }
        if (b_out) b_out[o] = (o < normal && b_in) ? b_in[o] : 0.f;
    }
    return CTC_OK;
}

ctc_status ctc_threshold_from_samples(const double *S, int64_t n, double alpha,
                                      double *ref, double *tau) {
    if (!S || !ref || !tau || n < 1 || !(alpha >= 0.0 && alpha <= 1.0))
        return fail(CTC_ERR_ARG, "bad threshold arguments");
    double sum = 0.0;
    for (int64_t i = 0; i < n; i++) sum += S[i];
    const double r = sum / (double)n;
    std::vector<double> dev(n);
    for (int64_t i = 0; i < n; i++) dev[i] = std::fabs(S[i] - r);
    std::sort(dev.begin(), dev.end());
    int64_t k = n - (int64_t)std::ceil(alpha * (double)n - 1e-12) + 1;
    k = std::min<int64_t>(std::max<int64_t>(k, 1), n);
    *ref = r;
    *tau = dev[k - 1];
    return CTC_OK;
}

ctc_status ctc_threshold_at_ref(const double *S, int64_t n, double ref,
                                double alpha, double *tau) {
    if (!S || !tau || n < 1 || !(alpha >= 0.0 && alpha <= 1.0) ||
        std::isnan(ref))
        return fail(CTC_ERR_ARG, "bad threshold arguments");
    std::vector<double> dev(n);
    for (int64_t i = 0; i < n; i++) {
        const double d = std::fabs(S[i] - ref);
        dev[i] = std::isnan(d) ? HUGE_VAL : d;
    }
    std::sort(dev.begin(), dev.end());
    int64_t k = n - (int64_t)std::ceil(alpha * (double)n - 1e-12) + 1;
    k = std::min<int64_t>(std::max<int64_t>(k, 1), n);
    *tau = dev[k - 1];
    return CTC_OK;
}

// ---------------------------------------------------------------------------
// L1-norm choice of the pruned channel (Sec. II-A): channel groups, norms,
// swap of the chosen channel with the last one.
// ---------------------------------------------------------------------------
namespace {

struct Dsu {
    std::vector<int> p;
    explicit Dsu(int n) : p(n) { for (int i = 0; i < n; i++) p[i] = i; }
    int find(int a) { while (p[a] != a) a = p[a]; return a; }
    void unite(int a, int b) {
        a = find(a); b = find(b);
        if (a != b) p[std::max(a, b)] = std::min(a, b);
    }
};

// channel count of tensor t (0 = input, i+1 = output of op i); -1 unknown
int tensor_channels(const ctc_op *ops, int n_ops, int t, int depth = 0) {
    if (t == 0 || depth > n_ops) return -1;
    const ctc_op &o = ops[t - 1];
    if (o.kind == CTC_OP_CONV || o.kind == CTC_OP_FC) return o.c_out;
    return tensor_channels(ops, n_ops, o.input, depth + 1);  // pooling
}

}  // namespace

ctc_status ctc_select_channels_l1(const ctc_op *ops, int32_t n_ops,
                                  float *const *params, int32_t *chosen) {
    if (!ops || n_ops < 1 || !params) return fail(CTC_ERR_ARG, "bad select arguments");
    const int nt = n_ops + 1;
    for (int i = 0; i < n_ops; i++) {
        const ctc_op &o = ops[i];
        if (o.input < 0 || o.input > i || o.residual > i ||
            o.kind < CTC_OP_CONV || o.kind > CTC_OP_FC)
            return fail(CTC_ERR_ARG, "op %d: bad tensor ids or kind", i);
        if ((o.kind == CTC_OP_CONV || o.kind == CTC_OP_FC) &&
            (!params[6 * i] || o.c_in < 1 || o.c_out < 1 ||
             (o.kind == CTC_OP_CONV && (o.k < 1 || o.groups < 1 ||
                                        o.c_in % o.groups))))
            return fail(CTC_ERR_ARG, "op %d: missing weights or bad shape", i);
    }
    Dsu dsu(nt);
    for (int i = 0; i < n_ops; i++) {
        const ctc_op &o = ops[i];
        if (o.kind == CTC_OP_CONV) {
            if (o.groups > 1) dsu.unite(o.input, i + 1);
            if (o.residual >= 0) dsu.unite(i + 1, o.residual);
        } else if (o.kind == CTC_OP_MAXPOOL || o.kind == CTC_OP_GAP) {
            dsu.unite(o.input, i + 1);
        }
    }
    std::vector<int> grp(nt);
    for (int t = 0; t < nt; t++) grp[t] = dsu.find(t);
    // channel count of every group (all its tensors must agree)
    std::vector<int> gch(nt, -1);
    for (int t = 1; t < nt; t++) {
        const int c = tensor_channels(ops, n_ops, t);
        if (c < 0) continue;
        int &g = gch[grp[t]];
        if (g >= 0 && g != c)
            return fail(CTC_ERR_ARG, "tensor %d: channels disagree in its group", t);
        g = c;
    }
    std::vector<std::vector<double>> imp(nt);
    std::vector<char> produced(nt, 0);
    auto add = [&](int g, const std::vector<double> &v) -> bool {
        if (gch[g] >= 0 && (int)v.size() != gch[g]) return false;
        if (imp[g].empty()) imp[g].assign(v.size(), 0.0);
        if (imp[g].size() != v.size()) return false;
        for (size_t c = 0; c < v.size(); c++) imp[g][c] += v[c];
        return true;
    };
    for (int i = 0; i < n_ops; i++) {
        const ctc_op &o = ops[i];
        const float *w = params[6 * i];
        if (o.kind == CTC_OP_CONV) {
            const int K = o.c_out, Cg = o.c_in / o.groups, RS = o.k * o.k;
            const int row = Cg * RS;
            std::vector<double> pv(K, 0.0);
            for (int k = 0; k < K; k++) {
                double a = 0.0;
                for (int j = 0; j < row; j++) a += std::fabs((double)w[(size_t)k * row + j]);
                pv[k] = a;
            }
            if (!add(grp[i + 1], pv)) return fail(CTC_ERR_ARG, "op %d: group size", i);
            produced[grp[i + 1]] = 1;
            if (o.groups == 1) {
                std::vector<double> cv(Cg, 0.0);
                for (int c = 0; c < Cg; c++) {
                    double a = 0.0;
                    for (int k = 0; k < K; k++)
                        for (int j = 0; j < RS; j++)
                            a += std::fabs((double)w[((size_t)k * Cg + c) * RS + j]);
                    cv[c] = a;
                }
                if (o.input > 0 && !add(grp[o.input], cv))
                    return fail(CTC_ERR_ARG, "op %d: input group size", i);
            }
        } else if (o.kind == CTC_OP_FC) {
            const int O = o.c_out, I = o.c_in;
            if (!o.final_fc) {
                std::vector<double> pv(O, 0.0);
                for (int r = 0; r < O; r++) {
                    double a = 0.0;
                    for (int j = 0; j < I; j++) a += std::fabs((double)w[(size_t)r * I + j]);
                    pv[r] = a;
                }
                if (!add(grp[i + 1], pv)) return fail(CTC_ERR_ARG, "op %d: group size", i);
                produced[grp[i + 1]] = 1;
            }
            std::vector<double> cv;
            if (o.flatten_c > 0) {
                const int C = o.flatten_c, HW = o.flatten_h * o.flatten_w;
                if (C * HW != I) return fail(CTC_ERR_ARG, "op %d: flatten shape", i);
                cv.assign(C, 0.0);
                for (int c = 0; c < C; c++) {
                    double a = 0.0;
                    for (int r = 0; r < O; r++)
                        for (int j = 0; j < HW; j++)
                            a += std::fabs((double)w[(size_t)r * I + (size_t)c * HW + j]);
                    cv[c] = a;
                }
            } else {
                cv.assign(I, 0.0);
                for (int f = 0; f < I; f++) {
                    double a = 0.0;
                    for (int r = 0; r < O; r++) a += std::fabs((double)w[(size_t)r * I + f]);
                    cv[f] = a;
                }
            }
            if (o.input > 0 && !add(grp[o.input], cv))
                return fail(CTC_ERR_ARG, "op %d: input group size", i);
        }
    }
    std::vector<int> pick(nt, -1);
    for (int g = 0; g < nt; g++) {
        if (!produced[g] || g == grp[0] || g == grp[n_ops] || imp[g].empty()) continue;
        pick[g] = (int)(std::min_element(imp[g].begin(), imp[g].end()) - imp[g].begin());
    }
    auto swap_rows = [](float *a, int n_rows, size_t row, int c, int last) {
        (void)n_rows;
        if (!a || c == last) return;
        for (size_t j = 0; j < row; j++) std::swap(a[(size_t)c * row + j], a[(size_t)last * row + j]);
    };
    for (int i = 0; i < n_ops; i++) {
        const ctc_op &o = ops[i];
        float *const *pp = params + 6 * i;
        if (o.kind == CTC_OP_CONV) {
            const int K = o.c_out, Cg = o.c_in / o.groups, RS = o.k * o.k;
            const int c = pick[grp[i + 1]];
            if (c >= 0 && c != K - 1) {
                swap_rows(pp[0], K, (size_t)Cg * RS, c, K - 1);
                for (int q = 1; q < 6; q++) swap_rows(pp[q], K, 1, c, K - 1);
            }
            const int ci = o.input > 0 ? pick[grp[o.input]] : -1;
            if (o.groups == 1 && ci >= 0 && ci != Cg - 1)
                for (int k = 0; k < K; k++)
                    for (int j = 0; j < RS; j++)
                        std::swap(pp[0][((size_t)k * Cg + ci) * RS + j],
                                  pp[0][((size_t)k * Cg + Cg - 1) * RS + j]);
        } else if (o.kind == CTC_OP_FC) {
            const int O = o.c_out, I = o.c_in;
            const int c = o.final_fc ? -1 : pick[grp[i + 1]];
            if (c >= 0 && c != O - 1) {
                swap_rows(pp[0], O, (size_t)I, c, O - 1);
                for (int q = 1; q < 6; q++) swap_rows(pp[q], O, 1, c, O - 1);
            }
            const int ci = o.input > 0 ? pick[grp[o.input]] : -1;
            if (ci >= 0) {
                const int C = o.flatten_c > 0 ? o.flatten_c : I;
                const int HW = o.flatten_c > 0 ? o.flatten_h * o.flatten_w : 1;
                if (ci != C - 1)
                    for (int r = 0; r < O; r++)
                        for (int j = 0; j < HW; j++)
                            std::swap(pp[0][(size_t)r * I + (size_t)ci * HW + j],
                                      pp[0][(size_t)r * I + (size_t)(C - 1) * HW + j]);
            }
        }
    }
    if (chosen)
        for (int i = 0; i < n_ops; i++) chosen[i] = pick[grp[i + 1]];
    return CTC_OK;
}

// The arguments of a standalone conv (ctc_conv2d_forward and its
// workspace query), validated.
static ctc_status conv2d_args(const ctc_layer_desc *d, ctc_dtype dtype, int32_t n,
                              int32_t h, int32_t w, int32_t relu, int32_t pool,
                              ConvArgs &a) {
    ctc_status s = validate_desc(d);
    if (s != CTC_OK) return s;
    if (dtype != CTC_F32 && dtype != CTC_F16)
        return fail(CTC_ERR_ARG, "bad dtype");
    if (n < 0 || h < 1 || w < 1) return fail(CTC_ERR_ARG, "bad conv2d sizes");
    if (d->c_in % 4 || d->c_out % 4)
        return fail(CTC_ERR_UNSUPPORTED, "channel counts must be multiples of 4");
    if (d->kh != d->kw) return fail(CTC_ERR_UNSUPPORTED, "square kernels only");
    const int P = (h + 2 * d->pad - d->kh) / d->stride + 1;
    const int Q = (w + 2 * d->pad - d->kw) / d->stride + 1;
    if (P < 1 || Q < 1) return fail(CTC_ERR_ARG, "empty output");
    if (pool != 0 && pool != 2) return fail(CTC_ERR_ARG, "pool must be 0 or 2");
    a = ConvArgs{};
    a.nimg = n; a.H = h; a.W = w; a.Cs = d->c_in; a.P = P; a.Q = Q;
    a.N = d->c_out; a.R = d->kh; a.S = d->kw; a.stride = d->stride;
    a.pad = d->pad; a.relu = relu; a.pool = pool;
    if (d->groups > 1 && dtype == CTC_F16 && d->c_out % 8)
        return fail(CTC_ERR_UNSUPPORTED, "fp16 depthwise needs channels %% 8");
    if (pool && (d->groups > 1 || !conv_pool_ok(dtype, a)))
        return fail(CTC_ERR_UNSUPPORTED, "no fused 2x2 max pool for this conv");
    return CTC_OK;
}

// fp32 partial sums of the split-K layers: ranges x output elements
static size_t conv2d_part_bytes(ctc_dtype dtype, const ConvArgs &a, int groups) {
    if (groups > 1 || a.pool || choose_tile(dtype, a).IMW > 0) return 0;
    const int sk = conv_splitk(dtype, a);
    return sk > 1 ? (size_t)sk * a.nimg * a.P * a.Q * a.N * 4 : 0;
}

ctc_status ctc_conv2d_workspace_bytes(const ctc_layer_desc *d, ctc_dtype dtype,
                                      int32_t n, int32_t h, int32_t w,
                                      int32_t pool, size_t *bytes) {
    if (!bytes) return fail(CTC_ERR_ARG, "NULL bytes");
    ConvArgs a;
    ctc_status s = conv2d_args(d, dtype, n, h, w, 0, pool, a);
    if (s != CTC_OK) return s;
    *bytes = conv2d_part_bytes(dtype, a, d->groups);
    return CTC_OK;
}

ctc_status ctc_conv2d_kernel_name(const ctc_layer_desc *d, ctc_dtype dtype,
                                  int32_t n, int32_t h, int32_t w, int32_t pool,
                                  char *name, int32_t cap) {
    if (!name || cap < 1) return fail(CTC_ERR_ARG, "bad name buffer");
    ConvArgs a;
    ctc_status s = conv2d_args(d, dtype, n, h, w, 1, pool, a);
    if (s != CTC_OK) return s;
    std::string k;
    if (d->groups > 1) k = dwconv_kernel_name(dtype, a);
    else if (pool) k = conv_kernel_name(dtype, a);
    else {
        TileCfg tc = choose_tile(dtype, a);
        k = tc.IMW > 0 ? conv_tile_name(dtype, tc) : conv_kernel_name(dtype, a);
    }
    snprintf(name, cap, "%s", k.c_str());
    return CTC_OK;
}

ctc_status ctc_conv2d_forward(const ctc_layer_desc *d, ctc_dtype dtype,
                              int32_t n, int32_t h, int32_t w,
                              const void *x, const void *wp,
                              const float *scale, const float *shift,
                              const void *residual, int32_t relu, int32_t pool,
                              void *y, void *workspace, size_t ws_bytes,
                              void *stream) {
    ConvArgs a;
    ctc_status s = conv2d_args(d, dtype, n, h, w, relu, pool, a);
    if (s != CTC_OK) return s;
    if (!x || !wp || !scale || !shift || !y)
        return fail(CTC_ERR_ARG, "bad conv2d_forward arguments");
    if (ws_bytes && !workspace) return fail(CTC_ERR_ARG, "ws_bytes without workspace");
    a.x = x; a.w = wp; a.scale = scale; a.shift = shift; a.res = residual;
    a.y = y;
    // split K over the caller's workspace when it holds the partial sums
    const size_t need = conv2d_part_bytes(dtype, a, d->groups);
    if (need && workspace && ws_bytes >= need) a.part = (float *)workspace;
    hipError_t e = d->groups > 1 ? launch_dwconv(dtype, a, S(stream))
                                 : launch_any_conv(dtype, a, S(stream));
    if (e != hipSuccess) return fail(CTC_ERR_DEVICE, "%s", hipGetErrorString(e));
    return CTC_OK;
}

ctc_status ctc_conv2d_forward_noalloc(const ctc_layer_desc *d, ctc_dtype dtype,
                                      int32_t n, int32_t h, int32_t w,
                                      const void *x, const void *wp,
                                      const float *scale, const float *shift,
                                      const void *residual, int32_t relu,
                                      int32_t pool, void *y, void *stream) {
    ConvArgs a;
    ctc_status s = conv2d_args(d, dtype, n, h, w, relu, pool, a);
    if (s != CTC_OK) return s;
    if (!x || !wp || !scale || !shift || !y)
        return fail(CTC_ERR_ARG, "bad conv2d_forward_noalloc arguments");
    a.x = x; a.w = wp; a.scale = scale; a.shift = shift; a.res = residual;
    a.y = y;
    const size_t need = conv2d_part_bytes(dtype, a, d->groups);
    if (need > conv_scratch_bytes())
        return fail(CTC_ERR_WORKSPACE,
                    "split-K partial sums need %zu bytes, beyond the %zu-byte "
                    "static scratch (use ctc_conv2d_forward with a workspace)",
                    need, conv_scratch_bytes());
    if (need) {
        // every k range writes its whole partial-sum block before the
        // reduction reads it: nothing in the scratch must start at zero
        void *p = nullptr;
        hipError_t e = conv_scratch(&p);
        if (e != hipSuccess)
            return fail(CTC_ERR_DEVICE, "scratch address: %s", hipGetErrorString(e));
        a.part = (float *)p;
    }
    hipError_t e = d->groups > 1 ? launch_dwconv(dtype, a, S(stream))
                                 : launch_any_conv(dtype, a, S(stream));
    if (e != hipSuccess) return fail(CTC_ERR_DEVICE, "%s", hipGetErrorString(e));
    return CTC_OK;
}

ctc_status ctc_verify(const float *Sv, int32_t batch, int32_t stride,
                      float ref, float tau, uint8_t *flags,
                      int32_t *n_flagged, int32_t *idx, void *stream) {
    if (!Sv || !n_flagged || batch < 1 || batch > 4096 || stride < 1)
        return fail(CTC_ERR_ARG, "bad verify arguments");
    HIP_TRY(launch_verify(Sv, batch, stride, ref, tau, flags, n_flagged, idx,
                          S(stream)));
    return CTC_OK;
}

static ctc_status create_impl(const ctc_op *ops, int32_t n_ops, int32_t in_c,
                              int32_t in_h, int32_t in_w, int32_t classes,
                              ctc_dtype dtype, int32_t protect, ctc_net **out) {
    if (!ops || n_ops < 1 || !out || in_c < 1 || in_h < 1 || in_w < 1 ||
        classes < 1)
        return fail(CTC_ERR_ARG, "bad net_create arguments");
    if (in_c > 4) return fail(CTC_ERR_UNSUPPORTED, "input with more than 4 channels");
    if (dtype != CTC_F32 && dtype != CTC_F16) return fail(CTC_ERR_ARG, "bad dtype");
    ctc_net *net = new ctc_net();
    net->in_c = in_c; net->in_h = in_h; net->in_w = in_w;
    net->classes = classes; net->dt = dtype; net->protect = protect ? 1 : 0;
    net->t.resize(n_ops);
    TensorInfo &t0 = net->t[0];
    // input staged NHWC with 4 channels (3 + zero) in both dtypes: the
    // stems (K = 27..147) run fastest on conv_igemm's 4-channel path
    t0.c = in_c; t0.h = in_h; t0.w = in_w; t0.cs = 4; t0.dt = dtype;
    auto bad = [&](ctc_status s, const char *fmt, int i) {
        delete net;
        return fail(s, fmt, i);
    };
    for (int i = 0; i < n_ops; i++) {
        OpPlan op;
        op.spec = ops[i];
        const ctc_op &o = op.spec;
        if (o.input < 0 || o.input > i) return bad(CTC_ERR_ARG, "op %d: bad input", i);
        const TensorInfo &ti = net->t[o.input];
        const bool last = i == n_ops - 1;
        if (last != (o.kind == CTC_OP_FC && o.final_fc))
            return bad(CTC_ERR_UNSUPPORTED, "op %d: the last op must be the final FC", i);
        TensorInfo to;
        if (o.kind == CTC_OP_CONV) {
            if (o.c_in != ti.c || o.k < 1 || o.stride < 1 || o.pad < 0 ||
                o.groups < 1 || o.c_in % o.groups)
                return bad(CTC_ERR_ARG, "op %d: conv shape mismatch", i);
            if (o.c_out % 4) return bad(CTC_ERR_UNSUPPORTED, "op %d: c_out %% 4", i);
            op.dw = o.groups > 1;
            if (op.dw && !(o.groups == o.c_in && o.c_in == o.c_out))
                return bad(CTC_ERR_UNSUPPORTED, "op %d: grouped conv must be depthwise", i);
            if (op.dw && dtype == CTC_F16 && o.c_out % 8)
                return bad(CTC_ERR_UNSUPPORTED, "op %d: fp16 depthwise needs channels %% 8", i);
            if (protect && o.k % 2 == 0)
                return bad(CTC_ERR_UNSUPPORTED, "op %d: even kernel", i);
            to.c = o.c_out; to.cs = o.c_out;
            to.h = (ti.h + 2 * o.pad - o.k) / o.stride + 1;
            to.w = (ti.w + 2 * o.pad - o.k) / o.stride + 1;
            if (to.h < 1 || to.w < 1) return bad(CTC_ERR_ARG, "op %d: empty output", i);
            to.dt = dtype;
            if (o.residual >= 0) {
                if (o.residual > i) return bad(CTC_ERR_ARG, "op %d: residual", i);
                const TensorInfo &tr = net->t[o.residual];
                if (tr.c != to.c || tr.h != to.h || tr.w != to.w || tr.dt != to.dt)
                    return bad(CTC_ERR_ARG, "op %d: residual shape", i);
            }
            op.role = protect ? derive_role(o) : CTC_ROLE_NONE;
            op.in_has_ck = protect && o.input != 0;
            op.n_out = o.c_out;
            op.ktot = op.dw ? o.k * o.k : o.k * o.k * ti.cs;
        } else if (o.kind == CTC_OP_MAXPOOL) {
            if (o.k < 1 || o.stride < 1 || o.pad < 0 || 2 * o.pad > o.k)
                return bad(CTC_ERR_ARG, "op %d: pool shape", i);
            to = ti;
            to.h = (ti.h + 2 * o.pad - o.k) / o.stride + 1;
            to.w = (ti.w + 2 * o.pad - o.k) / o.stride + 1;
            if (to.h < 1 || to.w < 1) return bad(CTC_ERR_ARG, "op %d: empty output", i);
        } else if (o.kind == CTC_OP_GAP) {
            to = ti;
            to.h = 1; to.w = 1;
        } else if (o.kind == CTC_OP_FC) {
            const int feat = ti.c * ti.h * ti.w;
            if (o.c_in != feat || ti.cs != ti.c)
                return bad(CTC_ERR_ARG, "op %d: FC input size", i);
            if (o.flatten_c > 0 &&
                (o.flatten_c != ti.c || o.flatten_h != ti.h || o.flatten_w != ti.w))
                return bad(CTC_ERR_ARG, "op %d: flatten shape", i);
            if (o.flatten_c == 0 && (ti.h != 1 || ti.w != 1))
                return bad(CTC_ERR_ARG, "op %d: FC on a map needs flatten", i);
            if (o.c_in % 4) return bad(CTC_ERR_UNSUPPORTED, "op %d: FC in %% 4", i);
            // fp16 activations are read 8 to a 16-byte load
            if (ti.dt == DT_F16 && o.c_in % 8)
                return bad(CTC_ERR_UNSUPPORTED, "op %d: fp16 FC in %% 8", i);
            op.rows = o.c_out + ((last && protect) ? 1 : 0);
            op.n_out = op.rows;
            op.in_has_ck = protect && o.input != 0;
            if (!last) {
                if (o.c_out % 4) return bad(CTC_ERR_UNSUPPORTED, "op %d: FC out %% 4", i);
                to.c = o.c_out; to.cs = o.c_out; to.h = 1; to.w = 1;
                to.dt = (o.out_f32 || (int)dtype == DT_F32) ? DT_F32 : DT_F16;
            } else if (o.c_out != classes) {
                return bad(CTC_ERR_ARG, "op %d: classes mismatch", i);
            }
        } else {
            return bad(CTC_ERR_ARG, "op %d: unknown kind", i);
        }
        if (!last) {
            to.img_elems = (size_t)to.h * to.w * to.cs;
            to.img_bytes = to.img_elems * (to.dt == DT_F16 ? 2 : 4);
            net->t[i + 1] = to;
        }
        net->ops.push_back(std::move(op));
    }
    // fusable inverted-residual blocks (fp16): expand 1x1 + ReLU ->
    // depthwise 3x3 pad 1 + ReLU -> project 1x1 (+ the block input), the two
    // intermediate tensors read by nothing else
    if (dtype == CTC_F16) {
        std::vector<int> readers(n_ops + 1, 0);
        for (int i = 0; i < n_ops; i++) {
            readers[net->ops[i].spec.input]++;
            if (net->ops[i].spec.residual >= 0) readers[net->ops[i].spec.residual]++;
        }
        // a 7x7 stride-2 stem whose output only feeds a 3x3 / 2 max pool
        for (int i = 0; i + 1 < n_ops; i++) {
            const OpPlan &c = net->ops[i], &m = net->ops[i + 1];
            const ctc_op &co = c.spec, &mo = m.spec;
            if (co.kind != CTC_OP_CONV || c.dw || mo.kind != CTC_OP_MAXPOOL ||
                mo.input != i + 1 || readers[i + 1] != 1 || mo.k != 3 || mo.stride != 2 ||
                mo.pad != 1 || co.residual >= 0)
                continue;
            const TensorInfo &tx = net->t[co.input], &ts = net->t[i + 1], &tp = net->t[i + 2];
            ConvArgs a{};
            a.nimg = 1; a.H = tx.h; a.W = tx.w; a.Cs = tx.cs; a.P = ts.h; a.Q = ts.w;
            a.N = co.c_out; a.R = co.k; a.S = co.k; a.stride = co.stride; a.pad = co.pad;
            if (tx.dt != DT_F16 || ts.cs != co.c_out || !stem_pool_ok(DT_F16, a, tp.h, tp.w))
                continue;
            net->ops[i].fuse = 7;
        }
        for (int i = 0; i + 2 < n_ops; i++) {
            const OpPlan &e = net->ops[i], &d = net->ops[i + 1], &pj = net->ops[i + 2];
            const ctc_op &eo = e.spec, &dd = d.spec, &po = pj.spec;
            if (eo.kind != CTC_OP_CONV || dd.kind != CTC_OP_CONV || po.kind != CTC_OP_CONV)
                continue;
            if (e.dw || eo.k != 1 || eo.stride != 1 || eo.pad != 0 || eo.residual >= 0 || !eo.relu)
                continue;
            if (!d.dw || dd.k != 3 || dd.pad != 1 || (dd.stride != 1 && dd.stride != 2) ||
                dd.residual >= 0 || !dd.relu || dd.input != i + 1)
                continue;
            if (pj.dw || po.k != 1 || po.stride != 1 || po.pad != 0 || po.input != i + 2)
                continue;
            if (po.residual >= 0 && (po.residual != eo.input || dd.stride != 1)) continue;
            if (readers[i + 1] != 1 || readers[i + 2] != 1) continue;
            const TensorInfo &tx = net->t[eo.input], &tdo = net->t[i + 2];
            IrArgs a{};
            a.nimg = 1; a.H = tx.h; a.W = tx.w; a.C = tx.cs; a.E = eo.c_out;
            a.Co = po.c_out; a.P = tdo.h; a.Q = tdo.w; a.stride = dd.stride;
            if (tx.dt != DT_F16 || tx.cs != tx.c || !ir_supported(a) || !ir_profitable(a))
                continue;
            net->ops[i].fuse = 3;
            i += 2;
        }
        // a block without an expand conv: depthwise 3x3 stride 1 pad 1 ->
        // pointwise 1x1, the depthwise output read by nothing else
        for (int i = 0; i + 1 < n_ops; i++) {
            if ((i >= 1 && net->ops[i - 1].fuse == 3) || (i >= 2 && net->ops[i - 2].fuse == 3))
                continue;                   // inside a fused three-op block
            const OpPlan &d = net->ops[i], &pj = net->ops[i + 1];
            const ctc_op &dd = d.spec, &po = pj.spec;
            if (d.fuse != 0 || dd.kind != CTC_OP_CONV || po.kind != CTC_OP_CONV) continue;
            if (!d.dw || dd.k != 3 || dd.stride != 1 || dd.pad != 1 || dd.residual >= 0)
                continue;
            if (pj.dw || po.k != 1 || po.stride != 1 || po.pad != 0 || po.input != i + 1 ||
                readers[i + 1] != 1)
                continue;
            const TensorInfo &tx = net->t[dd.input];
            DwPwArgs a{};
            a.nimg = 1; a.H = tx.h; a.W = tx.w; a.C = tx.cs; a.Co = po.c_out;
            if (tx.dt != DT_F16 || tx.cs != tx.c || !dwpw_supported(a)) continue;
            net->ops[i].fuse = 9;
            i += 1;
        }
    }
    // a dense conv whose output feeds only a 2x2 stride-2 max pool (VGG):
    // the pool runs in the conv's epilogue where its kernel supports it
    {
        std::vector<int> readers(n_ops + 1, 0);
        for (int i = 0; i < n_ops; i++) {
            readers[net->ops[i].spec.input]++;
            if (net->ops[i].spec.residual >= 0) readers[net->ops[i].spec.residual]++;
        }
        for (int i = 0; i + 1 < n_ops; i++) {
            const OpPlan &c = net->ops[i], &m = net->ops[i + 1];
            const ctc_op &co = c.spec, &mo = m.spec;
            if (co.kind == CTC_OP_CONV && !c.dw && c.fuse == 0 &&
                mo.kind == CTC_OP_MAXPOOL && mo.input == i + 1 && readers[i + 1] == 1 &&
                mo.k == 2 && mo.stride == 2 && mo.pad == 0)
                net->ops[i].fuse = 8;
        }
    }
    // fusable basic blocks (fp32): identity blocks of 16, 32 or 64 channels
    // (conv 3x3 stride 1 pad 1 + ReLU -> conv 3x3 stride 1 pad 1 + the first
    // conv's input + ReLU, the tensor between them read by nothing else)
    // and downsampling blocks 16 -> 32 and 32 -> 64 channels
    if (dtype == CTC_F32) {
        std::vector<int> readers(n_ops + 1, 0);
        for (int i = 0; i < n_ops; i++) {
            readers[net->ops[i].spec.input]++;
            if (net->ops[i].spec.residual >= 0) readers[net->ops[i].spec.residual]++;
        }
        auto conv33 = [&](const OpPlan &o) {
            const ctc_op &c = o.spec;
            return c.kind == CTC_OP_CONV && !o.dw && c.k == 3 && c.stride == 1 &&
                   c.pad == 1 && c.relu && c.c_in == c.c_out &&
                   (c.c_out == 16 || c.c_out == 32 || c.c_out == 64);
        };
        auto conv = [&](const OpPlan &o, int k, int stride, int pad, bool relu) {
            const ctc_op &c = o.spec;
            return c.kind == CTC_OP_CONV && !o.dw && c.k == k && c.stride == stride &&
                   c.pad == pad && (c.relu != 0) == relu;
        };
        for (int i = 0; i + 1 < n_ops; i++) {
            const OpPlan &a = net->ops[i], &b = net->ops[i + 1];
            // downsampling block: conv 3x3 stride 2 + ReLU, projection
            // shortcut 1x1 stride 2 on the same input, conv 3x3 + shortcut
            // + ReLU; both internal tensors read once
            if (i + 2 < n_ops && conv(a, 3, 2, 1, true) && conv(b, 1, 2, 0, false) &&
                conv(net->ops[i + 2], 3, 1, 1, true)) {
                const ctc_op &x1 = a.spec, &xs = b.spec, &x2 = net->ops[i + 2].spec;
                const TensorInfo &tx = net->t[x1.input];
                const bool shape = (x1.c_in == 16 && x1.c_out == 32) ||
                                   (x1.c_in == 32 && x1.c_out == 64);
                if (shape && x1.residual < 0 && xs.residual < 0 && xs.input == x1.input &&
                    xs.c_out == x1.c_out && x2.input == i + 1 && x2.residual == i + 2 &&
                    x2.c_in == x1.c_out && x2.c_out == x1.c_out && readers[i + 1] == 1 &&
                    readers[i + 2] == 1 && tx.dt == DT_F32 && tx.cs == tx.c) {
                    net->ops[i].fuse = 4;
                    i += 2;
                    continue;
                }
            }
            if (!conv33(a) || !conv33(b) || a.spec.residual >= 0) continue;
            if (b.spec.input != i + 1 || b.spec.residual != a.spec.input ||
                a.spec.c_out != b.spec.c_out || readers[i + 1] != 1)
                continue;
            const TensorInfo &tx = net->t[a.spec.input];
            if (tx.dt != DT_F32 || tx.cs != tx.c) continue;
            net->ops[i].fuse = 2;
            i += 1;
        }
        // a stem (conv 3x3 stride 1 pad 1 + ReLU on the 4-channel staged
        // input, 16 outputs) whose output only feeds the fused identity
        // block right after it
        for (int i = 0; i + 2 < n_ops; i++) {
            const OpPlan &a = net->ops[i];
            const ctc_op &c = a.spec;
            if (a.fuse != 0 || net->ops[i + 1].fuse != 2 || !conv(a, 3, 1, 1, true) ||
                c.residual >= 0 || c.c_out != 16 || net->ops[i + 1].spec.input != i + 1 ||
                readers[i + 1] != 2)
                continue;
            const TensorInfo &tx = net->t[c.input];
            if (tx.dt != DT_F32 || tx.cs != 4) continue;
            net->ops[i].fuse = 5;
        }
        // GAP followed by a small FC on its output alone
        for (int i = 0; i + 1 < n_ops; i++) {
            const OpPlan &g = net->ops[i], &f = net->ops[i + 1];
            if (g.spec.kind != CTC_OP_GAP || f.spec.kind != CTC_OP_FC ||
                f.spec.input != i + 1 || readers[i + 1] != 1)
                continue;
            const TensorInfo &tx = net->t[g.spec.input];
            FcArgs fa{};
            fa.I = f.spec.c_in;
            fa.O = f.rows;
            if (tx.dt != DT_F32 || tx.cs != tx.c || fa.I != tx.c || !gap_fc_ok(fa)) continue;
            net->ops[i].fuse = 6;
        }
        // a 64-channel identity block whose output only feeds such a GAP
        for (int i = 0; i + 3 < n_ops; i++) {
            const OpPlan &b = net->ops[i], &g = net->ops[i + 2], &f = net->ops[i + 3];
            if (b.fuse == 2 && b.spec.c_out == 64 && g.fuse == 6 &&
                g.spec.input == i + 2 && readers[i + 2] == 1 && f.rows <= 16 &&
                f.spec.c_in == 64)
                net->ops[i].head = true;
        }
    }
    t0.img_elems = (size_t)in_h * in_w * t0.cs;
    t0.img_bytes = t0.img_elems * ((int)dtype == DT_F16 ? 2 : 4);
    net->out_cols = classes + net->protect;
    *out = net;
    return CTC_OK;
}

// Workspace offsets for batches of up to max_batch images; written into the
// plan only when `commit`.
static size_t layout(ctc_net *net, int max_batch, bool commit) {
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
    for (auto &op : net->ops) {
        if (op.spec.kind != CTC_OP_CONV && op.spec.kind != CTC_OP_FC) continue;
        size_t wb = weight_elems(net, op) * wbytes(net);
        size_t w_off = take(wb), sc = take(op.n_out * 4), sh = take(op.n_out * 4);
        if (commit) { op.w_bytes = wb; op.w_off = w_off; op.sc_off = sc; op.sh_off = sh; }
    }
    for (auto &t : net->t) {
        size_t o = take(t.img_bytes * (size_t)max_batch);
        if (commit) t.off = o;
    }
    const int slots = RING_BATCHES * max_batch;
    size_t ring = take(net->t[0].img_bytes * (size_t)slots);
    size_t rows = take(sizeof(RowEnt) * (size_t)max_batch);
    size_t cnt = take(sizeof(int) * (size_t)max_batch);
    size_t fdev = take((size_t)NPASS * max_batch);
    // partial sums of the split-K convs, the largest layer's at max_batch
    size_t pbytes = 0;
    for (int i = 0; i < (int)net->ops.size(); i++) {
        const OpPlan &op = net->ops[i];
        if (op.spec.kind != CTC_OP_CONV || op.dw) continue;
        const TensorInfo &ti = net->t[op.spec.input], &to = net->t[i + 1];
        ConvArgs a{};
        a.nimg = max_batch; a.H = ti.h; a.W = ti.w; a.Cs = ti.cs;
        a.P = to.h; a.Q = to.w; a.N = op.spec.c_out;
        a.R = op.spec.k; a.S = op.spec.k; a.stride = op.spec.stride; a.pad = op.spec.pad;
        const int sk = conv_splitk(to.dt, a);
        if (sk > 1)
            pbytes = std::max(pbytes, (size_t)sk * max_batch * a.P * a.Q * a.N * 4);
    }
    // and of the split-K FC layers (the same buffer: one layer at a time)
    for (int i = 0; i < (int)net->ops.size(); i++) {
        const OpPlan &op = net->ops[i];
        if (op.spec.kind != CTC_OP_FC) continue;
        FcArgs fa{};
        fa.nimg = max_batch; fa.I = op.spec.c_in; fa.O = op.rows;
        pbytes = std::max(pbytes, fc_part_bytes(net->dt, fa));
    }
    size_t part = pbytes ? take(pbytes) : 0;
    if (commit) {
        net->part_off = part;
        net->part_bytes = pbytes;
        net->ring_off = ring;
        net->rowsdev_off = rows;
        net->cnt_off = cnt;
        net->flagdev_off = fdev;
        net->ring_slots = slots;
        net->af_cap = 4 * max_batch + 1024;
    }
    return off;
}

ctc_status ctc_net_workspace_bytes(const ctc_net *net, int32_t max_batch,
                                   size_t *bytes) {
    if (!net || !bytes || max_batch < 1 || max_batch > 4096)
        return fail(CTC_ERR_ARG, "bad workspace arguments");
    *bytes = layout(const_cast<ctc_net *>(net), max_batch, false);
    return CTC_OK;
}

static ctc_status upload_op(ctc_net *net, int i, hipStream_t st) {
    OpPlan &op = net->ops[i];
    std::vector<char> buf;
    pack_weights(net, op, buf);
    HIP_TRY(hipMemcpyAsync(net->ws + op.w_off, buf.data(), buf.size(),
                           hipMemcpyHostToDevice, st));
    std::vector<float> sc, sh;
    fold(op, sc, sh);
    HIP_TRY(hipMemcpyAsync(net->ws + op.sc_off, sc.data(), sc.size() * 4,
                           hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(net->ws + op.sh_off, sh.data(), sh.size() * 4,
                           hipMemcpyHostToDevice, st));
    HIP_TRY(hipStreamSynchronize(st));
    return CTC_OK;
}

static ctc_status bind_impl(ctc_net *net, const float *const *hp,
                            void *workspace, size_t ws_bytes,
                            int32_t max_batch, void *stream) {
    if (!net || !hp || !workspace) return fail(CTC_ERR_ARG, "bad bind arguments");
    if (max_batch < 1 || max_batch > 4096) return fail(CTC_ERR_ARG, "max_batch");
    if ((uintptr_t)workspace % ALIGN) return fail(CTC_ERR_WORKSPACE, "workspace alignment");
    size_t need = layout(net, max_batch, true);
    if (ws_bytes < need)
        return fail(CTC_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
    net->ws = (char *)workspace;
    net->ws_bytes = ws_bytes;
    net->max_batch = max_batch;
    hipStream_t st = S(stream);
    for (int i = 0; i < (int)net->ops.size(); i++) {
        OpPlan &op = net->ops[i];
        const ctc_op &o = op.spec;
        const float *const *p = hp + 6 * i;
        if (o.kind != CTC_OP_CONV && o.kind != CTC_OP_FC) continue;
        if (!p[0]) return fail(CTC_ERR_ARG, "op %d: NULL weights", i);
        if (o.has_bias != (p[1] != nullptr))
            return fail(CTC_ERR_ARG, "op %d: bias presence", i);
        if (o.kind == CTC_OP_CONV) {
            if (o.has_bn != (p[2] && p[3] && p[4] && p[5]))
                return fail(CTC_ERR_ARG, "op %d: BN presence", i);
            const size_t n = (size_t)o.c_out * (o.c_in / o.groups) * o.k * o.k;
            op.w.assign(p[0], p[0] + n);
            op.b = p[1] ? std::vector<float>(p[1], p[1] + o.c_out) : std::vector<float>();
            if (o.has_bn) {
                op.mean.assign(p[2], p[2] + o.c_out);
                op.var.assign(p[3], p[3] + o.c_out);
                op.gamma.assign(p[4], p[4] + o.c_out);
                op.beta.assign(p[5], p[5] + o.c_out);
            } else {
                op.mean.clear(); op.var.clear(); op.gamma.clear(); op.beta.clear();
            }
            if (net->protect) {
                ctc_layer_desc d{o.c_in, o.c_out, o.k, o.k, o.stride, o.pad,
                                 o.groups, op.in_has_ck, op.role};
                ctc_status s = build_conv(&d, op.w.data(),
                                          op.b.empty() ? nullptr : op.b.data(),
                                          o.has_bn ? op.mean.data() : nullptr,
                                          o.has_bn ? op.var.data() : nullptr,
                                          o.has_bn ? op.gamma.data() : nullptr,
                                          o.has_bn ? op.beta.data() : nullptr);
                if (s != CTC_OK) return s;
            }
        } else {
            const size_t I = o.c_in;
            std::vector<float> w(p[0], p[0] + (size_t)o.c_out * I);
            std::vector<float> b = p[1] ? std::vector<float>(p[1], p[1] + o.c_out)
                                        : std::vector<float>();
            if (net->protect) {
                int ckf = 0, ckn = 0;
                if (op.in_has_ck) {
                    if (o.flatten_c > 0) {
                        ckn = o.flatten_h * o.flatten_w;
                        ckf = (o.flatten_c - 1) * ckn;
                    } else {
                        ckf = o.c_in - 1; ckn = 1;
                    }
                }
                op.w.assign((size_t)op.rows * I, 0.f);
                op.b.assign(op.rows, 0.f);
                ctc_status s = ctc_build_fc(o.c_in, o.c_out, ckf, ckn, o.final_fc,
                                            w.data(), b.empty() ? nullptr : b.data(),
                                            op.w.data(), op.b.data());
                if (s != CTC_OK) return s;
                if (b.empty()) op.b.clear();
            } else {
                op.w = w;
                op.b = b;
            }
        }
        if (net->dt == DT_F16) {      // deployed weights are fp16 values
            op.w16.resize(op.w.size());
            for (size_t j = 0; j < op.w.size(); j++) {
                op.w16[j] = f32_to_f16_bits(op.w[j]);   // RNE
                op.w[j] = bits_f32(f16_widen_bits(op.w16[j]));
            }
        }
        ctc_status s = upload_op(net, i, st);
        if (s != CTC_OK) return s;
    }
    // arrival counters of the fused block heads: zero between kernels
    {
        std::vector<int> zero(max_batch, 0);
        HIP_TRY(hipMemcpyAsync(net->ws + net->cnt_off, zero.data(),
                               sizeof(int) * zero.size(), hipMemcpyHostToDevice, st));
        HIP_TRY(hipStreamSynchronize(st));
    }
    // pass records: host tables the kernels read (pinned, device-mapped)
    for (int k = 0; k < NPASS; k++) {
        PassRec &p = net->pass[k];
        if (p.ev) { (void)hipEventDestroy(p.ev); p.ev = nullptr; }
        if (p.ev_flags) { (void)hipEventDestroy(p.ev_flags); p.ev_flags = nullptr; }
        for (void *q : {(void *)p.rows, (void *)p.stage, (void *)p.faults,
                        (void *)p.flagrow})
            if (q) (void)hipHostFree(q);
        p.rows = nullptr; p.stage = nullptr; p.faults = nullptr; p.flagrow = nullptr;
        HIP_TRY(hipEventCreateWithFlags(&p.ev, hipEventDisableTiming));
        HIP_TRY(hipEventCreateWithFlags(&p.ev_flags, hipEventDisableTiming));
        p.flagdev = (uint8_t *)net->ws + net->flagdev_off + (size_t)k * max_batch;
        HIP_TRY(hipHostMalloc((void **)&p.rows, sizeof(RowEnt) * max_batch,
                              hipHostMallocDefault));
        HIP_TRY(hipHostMalloc((void **)&p.stage, sizeof(StageEnt) * 2 * max_batch,
                              hipHostMallocDefault));
        HIP_TRY(hipHostMalloc((void **)&p.faults, sizeof(ActFault) * net->af_cap,
                              hipHostMallocDefault));
        HIP_TRY(hipHostMalloc((void **)&p.flagrow, (size_t)max_batch,
                              hipHostMallocDefault));
        p.recorded = p.harvest = p.has_ev = false;
        p.no = p.deliver = -1;
        p.items.clear();
    }
    net->undelivered.clear();
    net->last_ev = -1;
    net->npass = 0;
    net->ncall = 0;
    net->queue.clear();
    net->slot_busy.assign(net->ring_slots, 0);
    net->slot_cursor = 0;
    net->pfaults.clear();
    net->afaults.clear();
    net->af_by_image.assign(max_batch, {});
    net->bound = true;
    return CTC_OK;
}

// ---------------------------------------------------------------------------
// Append mode: every conv and hidden FC gets one more output channel (the
// carry-through channel), rounded up to whole 16-byte channel vectors of the
// dtype (4 fp32, 8 fp16); the original filters keep their places, the
// padding channels have zero filters and identity BN, and the usual
// construction then turns the last channel into the carry-through channel.
// Nothing is pruned: the normal channels compute the unmodified network.
// ---------------------------------------------------------------------------
static int round_up(int v, int a) { return (v + a - 1) / a * a; }

static ctc_status widen_ops(const ctc_op *ops, int n, int in_c, int dt,
                            std::vector<ctc_op> &wide) {
    const int A = dt == DT_F16 ? 8 : 4;
    std::vector<int> cw(n + 1, 0);               // widened channels per tensor
    cw[0] = in_c;
    wide.assign(ops, ops + n);
    for (int i = 0; i < n; i++) {
        const ctc_op &o = ops[i];
        ctc_op &w = wide[i];
        if (o.input < 0 || o.input > i) return fail(CTC_ERR_ARG, "op %d: bad input", i);
        const int ci = cw[o.input];
        if (o.kind == CTC_OP_CONV) {
            w.c_in = ci;
            if (o.groups > 1) {
                if (!(o.groups == o.c_in && o.c_in == o.c_out))
                    return fail(CTC_ERR_UNSUPPORTED, "op %d: grouped conv must be depthwise", i);
                w.groups = w.c_out = ci;
            } else {
                w.c_out = round_up(o.c_out + 1, A);
            }
            cw[i + 1] = w.c_out;
        } else if (o.kind == CTC_OP_FC) {
            if (o.flatten_c > 0) {
                w.flatten_c = ci;
                w.c_in = ci * o.flatten_h * o.flatten_w;
            } else {
                w.c_in = ci;
            }
            w.c_out = o.final_fc ? o.c_out : round_up(o.c_out + 1, A);
            cw[i + 1] = w.c_out;
        } else {
            cw[i + 1] = ci;
        }
    }
    return CTC_OK;
}

// widened canonical parameters of every op from the caller's
static ctc_status widen_params(const ctc_net *net, const float *const *hp,
                               std::vector<std::vector<float>> &store,
                               std::vector<const float *> &ptr) {
    const int n = (int)net->user_ops.size();
    store.assign(6 * n, std::vector<float>());
    ptr.assign(6 * n, nullptr);
    for (int i = 0; i < n; i++) {
        const ctc_op &u = net->user_ops[i];
        const ctc_op &w = net->ops[i].spec;
        const float *const *p = hp + 6 * i;
        if (u.kind != CTC_OP_CONV && u.kind != CTC_OP_FC) continue;
        if (!p[0]) return fail(CTC_ERR_ARG, "op %d: NULL weights", i);
        if (u.kind == CTC_OP_CONV) {
            const int K = u.c_out, Cg = u.c_in / u.groups, RS = u.k * u.k;
            const int K2 = w.c_out, Cg2 = w.c_in / w.groups;
            std::vector<float> &ww = store[6 * i];
            ww.assign((size_t)K2 * Cg2 * RS, 0.f);
            for (int k = 0; k < K; k++)
                for (int c = 0; c < Cg; c++)
                    for (int j = 0; j < RS; j++)
                        ww[((size_t)k * Cg2 + c) * RS + j] = p[0][((size_t)k * Cg + c) * RS + j];
            const float idv[6] = {0.f, 0.f, 0.f, 1.f, 1.f, 0.f};   // b, mean, var, gamma, beta
            for (int q = 1; q < 6; q++) {
                if (!p[q]) continue;
                store[6 * i + q].assign(K2, idv[q]);
                std::copy(p[q], p[q] + K, store[6 * i + q].begin());
            }
        } else {
            const int O = u.c_out, I = u.c_in, O2 = w.c_out, I2 = w.c_in;
            std::vector<float> &ww = store[6 * i];
            ww.assign((size_t)O2 * I2, 0.f);
            // after a flatten the widened channels come after the original
            // ones in NCHW feature order, so feature f keeps its index
            for (int o = 0; o < O; o++)
                std::copy(p[0] + (size_t)o * I, p[0] + (size_t)(o + 1) * I,
                          ww.begin() + (size_t)o * I2);
            if (p[1]) {
                store[6 * i + 1].assign(O2, 0.f);
                std::copy(p[1], p[1] + O, store[6 * i + 1].begin());
            }
        }
        for (int q = 0; q < 6; q++)
            if (!store[6 * i + q].empty()) ptr[6 * i + q] = store[6 * i + q].data();
    }
    return CTC_OK;
}

ctc_status ctc_net_create(const ctc_op *ops, int32_t n_ops, int32_t in_c,
                          int32_t in_h, int32_t in_w, int32_t classes,
                          ctc_dtype dtype, int32_t protect, ctc_net **out) {
    if (protect != CTC_PROTECT_APPEND)
        return create_impl(ops, n_ops, in_c, in_h, in_w, classes, dtype,
                           protect ? 1 : 0, out);
    if (!ops || n_ops < 1 || !out) return fail(CTC_ERR_ARG, "bad net_create arguments");
    std::vector<ctc_op> wide;
    ctc_status s = widen_ops(ops, n_ops, in_c, (int)dtype, wide);
    if (s != CTC_OK) return s;
    s = create_impl(wide.data(), n_ops, in_c, in_h, in_w, classes, dtype, 1, out);
    if (s != CTC_OK) return s;
    (*out)->append = true;
    (*out)->user_ops.assign(ops, ops + n_ops);
    return CTC_OK;
}

ctc_status ctc_net_bind(ctc_net *net, const float *const *hp, void *workspace,
                        size_t ws_bytes, int32_t max_batch, void *stream) {
    if (!net || !hp) return fail(CTC_ERR_ARG, "bad bind arguments");
    if (!net->append) return bind_impl(net, hp, workspace, ws_bytes, max_batch, stream);
    std::vector<std::vector<float>> store;
    std::vector<const float *> ptr;
    ctc_status s = widen_params(net, hp, store, ptr);
    if (s != CTC_OK) return s;
    return bind_impl(net, ptr.data(), workspace, ws_bytes, max_batch, stream);
}

ctc_status ctc_net_set_threshold(ctc_net *net, float ref, float tau) {
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    net->ref = ref;
    net->tau = tau;
    return CTC_OK;
}

ctc_status ctc_network_forward(ctc_net *net, int32_t batch, const float *x,
                               float *out, uint8_t *flags, int32_t reexec,
                               void *stream) {
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    if (batch < 0 || batch > net->max_batch)
        return fail(CTC_ERR_ARG, "batch %d outside 0..%d", batch, net->max_batch);
    if (batch > 0 && (!x || !out)) return fail(CTC_ERR_ARG, "NULL input/output");
    if (reexec < CTC_REEXEC_NONE || reexec > CTC_REEXEC_DEFERRED)
        return fail(CTC_ERR_ARG, "bad reexec mode");
    hipStream_t st = S(stream);
    const int cols = net->out_cols;
    ctc_status s;
    if (!net->protect || reexec == CTC_REEXEC_NONE) {
        // one pass over exactly this batch; flags written, nothing re-run
        if (batch == 0) return CTC_OK;
        PassRec *p;
        if ((s = next_pass(net, &p, st)) != CTC_OK) return s;
        for (int r = 0; r < batch; r++) {
            Item it{-1, out + (size_t)r * cols, flags ? flags + r : nullptr, r,
                    true, -1};
            p->items.push_back(it);
            p->rows[r] = RowEnt{(int64_t)(uintptr_t)it.out,
                                (int64_t)(uintptr_t)it.flags, -1, 1};
            p->stage[r] = StageEnt{r, -1, r, 0};
        }
        p->harvest = false;
        return run_pass(net, *p, batch, x, st);
    }
    // Re-executing modes.  Results of the pass two back feed the queue
    // (flagged images go to its front); fresh images are staged into the
    // ring and join the queue's back; every pass takes exactly `batch`
    // items, and an extra pass runs once the backlog reaches a batch.
    if (net->npass >= SETTLE_LAG) {
        s = settle(net, (int)((net->npass - SETTLE_LAG) % NPASS), st);
        if (s != CTC_OK) return s;
    }
    if (batch > 0) {
        const long call = net->ncall++;
        // The pass runs the queue's first q items and this call's first m
        // images.  Normally its input rows are a run of consecutive ring
        // slots: this call's images are converted straight into the run,
        // the queued ones copied in after them, and the first layer reads
        // the run, so a fresh image is written once.  With a fault armed on
        // the input (it must not reach the copy that a re-execution reads)
        // or no free run, images get single slots and the pass input is
        // assembled in tensor 0.
        int base = -1;
        if (!input_faults_armed(net)) {
            base = alloc_run(net, batch);
            if (base < 0) {                  // ring busy: drain completions
                if ((s = settle_all(net, st)) != CTC_OK) return s;
                base = alloc_run(net, batch);
            }
        }
        const int q = std::min((int)net->queue.size(), batch);
        const int m = batch - q;
        // single slots: this call's images that wait in the queue (every
        // image without a run)
        std::vector<int> slots(batch, -1);
        for (int j = base >= 0 ? m : 0; j < batch; j++) {
            slots[j] = alloc_slot(net);
            if (slots[j] < 0) {            // ring full: drain completions
                if ((s = settle_all(net, st)) != CTC_OK) return s;
                slots[j] = alloc_slot(net);
                if (slots[j] < 0)
                    return fail(CTC_ERR_STATE, "re-execution ring exhausted");
            }
        }
        PassRec *p;
        if ((s = next_pass(net, &p, st)) != CTC_OK) return s;
        int ns = 0;
        auto row = [&](int r, const Item &it) {
            p->items.push_back(it);
            p->rows[r] = RowEnt{(int64_t)(uintptr_t)it.out,
                                (int64_t)(uintptr_t)it.flags, it.slot, it.first};
        };
        auto fresh = [&](int j, int slot) {
            return Item{slot, out + (size_t)j * cols, flags ? flags + j : nullptr,
                        j, true, call};
        };
        if (base >= 0) {
            for (int j = 0; j < m; j++) {              // converted into the run
                row(j, fresh(j, base + j));
                p->stage[ns++] = StageEnt{j, -1, j, 0};
            }
            for (int r = m; r < batch; r++) {          // copied into the run
                Item it = net->queue.front();
                net->queue.pop_front();
                p->stage[ns++] = StageEnt{-1, it.slot, r, 0};
                it.old_slot = it.slot;
                it.slot = base + r;
                row(r, it);
            }
            for (int j = m; j < batch; j++) {          // staged, then queued
                net->queue.push_back(fresh(j, slots[j]));
                p->stage[ns++] = StageEnt{j, slots[j], -1, 0};
            }
        } else {
            for (int j = 0; j < batch; j++) net->queue.push_back(fresh(j, slots[j]));
            std::vector<int> row_of(batch, -1);
            for (int r = 0; r < batch; r++) {
                Item it = net->queue.front();
                net->queue.pop_front();
                row(r, it);
                const bool mine = it.first && it.call == call;
                if (mine) row_of[it.img] = r;
                else p->stage[ns++] = StageEnt{-1, it.slot, r, 0};
            }
            for (int j = 0; j < batch; j++)
                p->stage[ns++] = StageEnt{j, slots[j], row_of[j], 0};
        }
        p->harvest = true;
        char *in0 = base >= 0 ? net->ws + net->ring_off +
                                    (size_t)base * net->t[0].img_bytes
                              : nullptr;
        if ((s = run_pass(net, *p, ns, x, st, in0)) != CTC_OK) return s;
        while ((int)net->queue.size() >= batch)
            if ((s = run_queue_pass(net, batch, st)) != CTC_OK) return s;
    }
    if (reexec == CTC_REEXEC_SYNC) return ctc_network_flush(net, stream);
    return CTC_OK;
}

ctc_status ctc_network_flush(ctc_net *net, void *stream) {
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    hipStream_t st = S(stream);
    ctc_status s;
    // Settling first puts the re-runs of every pass in flight into the
    // queue, so they share a pass with the waiting images (one partial pass
    // instead of two); the loop ends when a settle queues nothing more.
    for (;;) {
        if ((s = settle_all(net, st)) != CTC_OK) return s;
        if (net->queue.empty()) break;
        while (!net->queue.empty())
            if ((s = run_queue_pass(net, net->max_batch, st)) != CTC_OK) return s;
    }
    return CTC_OK;
}

// ------------------------------------------------------------ HIP graphs

// A captured run of one-pass inferences (Sec. II-B).  The graph's kernels
// read its own pinned row and staging tables at replay time, so those live
// as long as the graph; the detector's flags go to a device buffer of the
// graph's own, from which a re-executing launch reads them.
struct ctc_graph {
    ctc_net *net = nullptr;
    int batch = 0, passes = 0;
    const float *x = nullptr;
    float *out = nullptr;
    std::vector<PassRec> recs;
    RowEnt *rows = nullptr;        // pinned [passes * batch]
    StageEnt *stage = nullptr;     // pinned [passes * batch]
    uint8_t *flagdev = nullptr;    // device [passes * batch]
    uint8_t *flaghost = nullptr;   // pinned [passes * batch]
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    hipEvent_t done = nullptr;

    ~ctc_graph() {
        // kernels of a replay still running may read the tables
        (void)hipDeviceSynchronize();
        if (exec) (void)hipGraphExecDestroy(exec);
        if (graph) (void)hipGraphDestroy(graph);
        if (done) (void)hipEventDestroy(done);
        if (rows) (void)hipHostFree(rows);
        if (stage) (void)hipHostFree(stage);
        if (flaghost) (void)hipHostFree(flaghost);
        if (flagdev) (void)hipFree(flagdev);
    }
};

namespace {

// Ends a capture on every path out of ctc_graph_create.
struct CaptureGuard {
    ctc_net *net;
    hipStream_t st = nullptr;
    bool open = false;
    ~CaptureGuard() {
        net->capture = false;
        if (open) {
            hipGraph_t g = nullptr;
            (void)hipStreamEndCapture(st, &g);
            if (g) (void)hipGraphDestroy(g);
        }
        if (st) (void)hipStreamDestroy(st);
    }
};

}  // namespace

ctc_status ctc_graph_create(ctc_net *net, int32_t batch, int32_t passes,
                            const float *x, float *out, uint8_t *flags,
                            ctc_graph **graph) {
    if (!graph) return fail(CTC_ERR_ARG, "NULL graph");
    *graph = nullptr;
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    if (batch < 1 || batch > net->max_batch)
        return fail(CTC_ERR_ARG, "batch %d outside 1..%d", batch, net->max_batch);
    if (passes < 1 || (long)passes * batch > CTC_GRAPH_MAX_IMAGES)
        return fail(CTC_ERR_ARG, "%d passes of %d images: outside 1..%d images",
                    passes, batch, CTC_GRAPH_MAX_IMAGES);
    if (!x || !out) return fail(CTC_ERR_ARG, "NULL input/output");
    if (net->prof) return fail(CTC_ERR_STATE, "per-op profiling is on");
    if (!net->afaults.empty())
        return fail(CTC_ERR_STATE, "activation faults are armed");
    std::unique_ptr<ctc_graph> g(new ctc_graph);
    g->net = net;
    g->batch = batch;
    g->passes = passes;
    g->x = x;
    g->out = out;
    const size_t n = (size_t)passes * batch;
    HIP_TRY(hipHostMalloc((void **)&g->rows, sizeof(RowEnt) * n, hipHostMallocDefault));
    HIP_TRY(hipHostMalloc((void **)&g->stage, sizeof(StageEnt) * n, hipHostMallocDefault));
    HIP_TRY(hipHostMalloc((void **)&g->flaghost, n, hipHostMallocDefault));
    HIP_TRY(hipMalloc((void **)&g->flagdev, n));
    HIP_TRY(hipEventCreateWithFlags(&g->done, hipEventDisableTiming));
    g->recs.resize(passes);
    const int cols = net->out_cols;
    const size_t img = (size_t)net->in_c * net->in_h * net->in_w;
    CaptureGuard cg{net};
    // captured on a stream of its own: the caller's may be the null stream,
    // which cannot be captured
    HIP_TRY(hipStreamCreateWithFlags(&cg.st, hipStreamNonBlocking));
    HIP_TRY(hipStreamBeginCapture(cg.st, hipStreamCaptureModeRelaxed));
    cg.open = true;
    net->capture = true;
    for (int k = 0; k < passes; k++) {
        PassRec &p = g->recs[k];
        const size_t b0 = (size_t)k * batch;
        p.rows = g->rows + b0;
        p.stage = g->stage + b0;
        p.flagdev = g->flagdev + b0;
        p.harvest = false;
        for (int r = 0; r < batch; r++) {
            Item it{-1, out + (b0 + r) * cols, flags ? flags + b0 + r : nullptr, -1,
                    true, -1};
            p.items.push_back(it);
            p.rows[r] = RowEnt{(int64_t)(uintptr_t)it.out,
                               (int64_t)(uintptr_t)it.flags, -1, 1};
            p.stage[r] = StageEnt{r, -1, r, 0};
        }
        ctc_status s = run_pass(net, p, batch, x + b0 * img, cg.st);
        if (s != CTC_OK) return s;
    }
    cg.open = false;
    HIP_TRY(hipStreamEndCapture(cg.st, &g->graph));
    HIP_TRY(hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0));
    *graph = g.release();
    return CTC_OK;
}

ctc_status ctc_graph_launch(ctc_graph *g, int32_t reexec, int32_t *n_flagged,
                            void *stream) {
    if (n_flagged) *n_flagged = 0;
    if (!g) return fail(CTC_ERR_ARG, "NULL graph");
    if (reexec != CTC_REEXEC_NONE && reexec != CTC_REEXEC_SYNC)
        return fail(CTC_ERR_ARG, "reexec must be CTC_REEXEC_NONE or CTC_REEXEC_SYNC");
    ctc_net *net = g->net;
    if (reexec == CTC_REEXEC_SYNC && !net->protect)
        return fail(CTC_ERR_STATE, "re-execution needs a protected net");
    hipStream_t st = S(stream);
    HIP_TRY(hipGraphLaunch(g->exec, st));
    if (reexec == CTC_REEXEC_NONE) return CTC_OK;
    const size_t n = (size_t)g->passes * g->batch;
    HIP_TRY(hipMemcpyAsync(g->flaghost, g->flagdev, n, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipEventRecord(g->done, st));
    HIP_TRY(hipEventSynchronize(g->done));
    std::vector<int> idx;
    for (size_t i = 0; i < n; i++)
        if (g->flaghost[i]) idx.push_back((int)i);
    if (n_flagged) *n_flagged = (int32_t)idx.size();
    if (idx.empty()) return CTC_OK;
    // Sec. II-B: every flagged image runs once more, its output row
    // overwritten; the re-run's own flag is not kept
    const int cols = net->out_cols;
    for (size_t b = 0; b < idx.size(); b += net->max_batch) {
        const int m = (int)std::min(idx.size() - b, (size_t)net->max_batch);
        PassRec *p;
        ctc_status s = next_pass(net, &p, st);
        if (s != CTC_OK) return s;
        for (int r = 0; r < m; r++) {
            float *row = g->out + (size_t)idx[b + r] * cols;
            p->items.push_back(Item{-1, row, nullptr, -1, false, -1});
            p->rows[r] = RowEnt{(int64_t)(uintptr_t)row, 0, -1, 0};
            p->stage[r] = StageEnt{idx[b + r], -1, r, 0};
        }
        p->harvest = false;
        if ((s = run_pass(net, *p, m, g->x, st)) != CTC_OK) return s;
    }
    HIP_TRY(hipEventRecord(g->done, st));
    HIP_TRY(hipEventSynchronize(g->done));
    return CTC_OK;
}

void ctc_graph_destroy(ctc_graph *g) { delete g; }

// ---------------------------------------------------------------- faults

static ctc_status param_ref(ctc_net *net, const ctc_fault &f, OpPlan **op,
                            std::vector<float> **vec, int *width) {
    if (f.layer < 0 || f.layer >= (int)net->ops.size())
        return fail(CTC_ERR_ARG, "fault layer %d", f.layer);
    OpPlan &o = net->ops[f.layer];
    std::vector<float> *v = nullptr;
    switch (f.site) {
    case CTC_SITE_WEIGHT: v = &o.w; break;
    case CTC_SITE_BIAS: v = &o.b; break;
    case CTC_SITE_BN_MEAN: v = &o.mean; break;
    case CTC_SITE_BN_VAR: v = &o.var; break;
    case CTC_SITE_BN_GAMMA: v = &o.gamma; break;
    case CTC_SITE_BN_BETA: v = &o.beta; break;
    default: return fail(CTC_ERR_ARG, "fault site %d", f.site);
    }
    if (v->empty() || f.index < 0 || (size_t)f.index >= v->size())
        return fail(CTC_ERR_ARG, "fault index %lld out of range", (long long)f.index);
    *width = (f.site == CTC_SITE_WEIGHT && net->dt == DT_F16) ? 16 : 32;
    if (f.bit < 0 || f.bit >= *width) return fail(CTC_ERR_ARG, "fault bit %d", f.bit);
    *op = &o;
    *vec = v;
    return CTC_OK;
}

// Flips the bit in the host copy and writes the affected device values.
static ctc_status flip_param(ctc_net *net, const ctc_fault &f, hipStream_t st) {
    OpPlan *op;
    std::vector<float> *v;
    int width;
    ctc_status s = param_ref(net, f, &op, &v, &width);
    if (s != CTC_OK) return s;
    float &val = (*v)[f.index];
    uint32_t bits;
    if (width == 16) {             // XOR the deployed binary16 pattern itself
        if (op->w16.size() != v->size())
            return fail(CTC_ERR_STATE, "fp16 weights without their patterns");
        uint16_t &h = op->w16[f.index];
        h ^= (uint16_t)(1u << f.bit);
        bits = h;
        val = bits_f32(f16_widen_bits(h));
    } else {
        bits = f32_bits(val) ^ (1u << f.bit);
        val = bits_f32(bits);
    }
    if (f.site == CTC_SITE_WEIGHT) {
        size_t p = packed_index(net, *op, f.index);
        char *addr = net->ws + op->w_off + p * (width / 8);
        HIP_TRY(launch_set_bits(addr, bits, width, st));
    } else {
        std::vector<float> sc, sh;
        fold(*op, sc, sh);
        const size_t k = f.index;
        HIP_TRY(launch_set_bits(net->ws + op->sc_off + 4 * k, f32_bits(sc[k]), 32, st));
        HIP_TRY(launch_set_bits(net->ws + op->sh_off + 4 * k, f32_bits(sh[k]), 32, st));
    }
    return CTC_OK;
}

ctc_status ctc_inject_bitflip(ctc_net *net, const ctc_fault *faults, int32_t n,
                              void *stream) {
    if (!net || (n > 0 && !faults) || n < 0) return fail(CTC_ERR_ARG, "bad inject arguments");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    hipStream_t st = S(stream);
    const int nops = (int)net->ops.size();
    // validate everything first
    for (int i = 0; i < n; i++) {
        const ctc_fault &f = faults[i];
        if (f.site == CTC_SITE_ACT) {
            if (f.layer < 0 || f.layer > nops) return fail(CTC_ERR_ARG, "act tensor %d", f.layer);
            if (f.image < 0 || f.image >= net->max_batch)
                return fail(CTC_ERR_ARG, "act image %d", f.image);
            int width;
            int64_t elems;
            if (f.layer == nops) { width = 32; elems = net->out_cols; }
            else {
                const TensorInfo &t = net->t[f.layer];
                width = t.dt == DT_F16 ? 16 : 32;
                elems = (int64_t)t.c * t.h * t.w;
            }
            if (f.index < 0 || f.index >= elems) return fail(CTC_ERR_ARG, "act index");
            if (f.bit < 0 || f.bit >= width) return fail(CTC_ERR_ARG, "act bit");
        } else {
            OpPlan *op;
            std::vector<float> *v;
            int width;
            ctc_status s = param_ref(net, f, &op, &v, &width);
            if (s != CTC_OK) return s;
        }
    }
    bool act = false;
    for (int i = 0; i < n; i++) {
        const ctc_fault &f = faults[i];
        if (f.site == CTC_SITE_ACT) {
            ActFault a{};
            a.image = f.image;
            a.bit = f.bit;
            if (f.layer == nops) {
                a.width = 32;
                a.offset = f.index * 4;
            } else {
                const TensorInfo &t = net->t[f.layer];
                int64_t hw = (int64_t)t.h * t.w;
                int64_t c = f.index / hw, p = f.index % hw;
                a.width = t.dt == DT_F16 ? 16 : 32;
                a.offset = (p * t.cs + c) * (a.width / 8);
            }
            if ((int)net->afaults.size() >= net->af_cap)
                return fail(CTC_ERR_ARG, "more than %d armed activation faults",
                            net->af_cap);
            net->af_by_image[f.image].push_back((int)net->afaults.size());
            net->afaults.push_back({f.layer, a});
            act = true;
        } else {
            ctc_status s = flip_param(net, f, st);
            if (s != CTC_OK) return s;
            net->pfaults.push_back({f});
        }
    }
    (void)act;
    return CTC_OK;
}

ctc_status ctc_clear_faults(ctc_net *net, void *stream) {
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    hipStream_t st = S(stream);
    for (auto it = net->pfaults.rbegin(); it != net->pfaults.rend(); ++it) {
        ctc_status s = flip_param(net, it->f, st);
        if (s != CTC_OK) return s;
    }
    net->pfaults.clear();
    net->afaults.clear();
    for (auto &v : net->af_by_image) v.clear();
    return CTC_OK;
}

ctc_status ctc_net_tensor(const ctc_net *net, int32_t t, void **dev,
                          int32_t *c_stored, int32_t *h, int32_t *w,
                          int32_t *dtype) {
    if (!net || t < 0 || t >= (int)net->t.size())
        return fail(CTC_ERR_ARG, "bad tensor id");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    const TensorInfo &ti = net->t[t];
    if (dev) *dev = net->ws + ti.off;
    if (c_stored) *c_stored = ti.cs;
    if (h) *h = ti.h;
    if (w) *w = ti.w;
    if (dtype) *dtype = ti.dt;
    return CTC_OK;
}

ctc_status ctc_net_weight_address(ctc_net *net, int32_t layer, int64_t index,
                                  void **dev, int32_t *bits) {
    if (!net || !dev || !bits) return fail(CTC_ERR_ARG, "NULL argument");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    ctc_fault f{};
    f.site = CTC_SITE_WEIGHT;
    f.layer = layer;
    f.index = index;
    OpPlan *op;
    std::vector<float> *v;
    int width;
    ctc_status s = param_ref(net, f, &op, &v, &width);
    if (s != CTC_OK) return s;
    *dev = net->ws + op->w_off + packed_index(net, *op, (size_t)index) * (width / 8);
    *bits = width;
    return CTC_OK;
}

ctc_status ctc_net_profile(ctc_net *net, int32_t enable) {
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    net->prof = enable != 0;
    net->prof_marks.resize(net->ops.size() + 2);
    return CTC_OK;
}

ctc_status ctc_net_profile_read(ctc_net *net, int32_t *launches,
                                double *total_ms) {
    if (!net || !launches || !total_ms) return fail(CTC_ERR_ARG, "bad profile_read");
    const size_t ns = net->ops.size() + 2;
    net->prof_marks.resize(ns);
    if (net->ev_used > 0) HIP_TRY(hipEventSynchronize(net->ev_pool[net->ev_used - 1]));
    for (size_t k = 0; k < ns; k++) {
        double tot = 0.0;
        for (auto &pr : net->prof_marks[k]) {
            float ms = 0.f;
            HIP_TRY(hipEventElapsedTime(&ms, net->ev_pool[pr.first],
                                        net->ev_pool[pr.second]));
            tot += ms;
        }
        launches[k] = (int32_t)net->prof_marks[k].size();
        total_ms[k] = tot;
        net->prof_marks[k].clear();
    }
    net->ev_used = 0;
    return CTC_OK;
}

ctc_status ctc_net_op_kernel(const ctc_net *net, int32_t i, int32_t nimg,
                             char *name, int32_t cap) {
    if (!net || !name || cap < 1 || i < 0 || i >= (int)net->ops.size())
        return fail(CTC_ERR_ARG, "bad op_kernel arguments");
    const OpPlan &op = net->ops[i];
    const ctc_op &o = op.spec;
    std::string s;
    const int dt = net->dt;
    const char *tn = dt == DT_F16 ? "_Float16" : "float";
    auto fc_name = [&](int j) {
        const OpPlan &fo = net->ops[j];
        FcArgs fa{};
        fa.nimg = nimg; fa.I = fo.spec.c_in; fa.O = fo.rows;
        const int dout = j == (int)net->ops.size() - 1 ? DT_F32 : net->t[j + 1].dt;
        return std::string(fc_kernel_name(net->t[fo.spec.input].dt, dt, dout, fa));
    };
    const bool stem_pool = (net->fusion & CTC_FUSE_STEM) &&
                           ((o.kind == CTC_OP_CONV && op.fuse == 7) ||
                            (o.kind == CTC_OP_MAXPOOL && i > 0 && net->ops[i - 1].fuse == 7));
    // a conv with the 2x2 max pool in its epilogue, and that pool
    const int pc = o.kind == CTC_OP_CONV ? i : i - 1;
    bool conv_pool = false;
    ConvArgs pa{};
    if ((net->fusion & CTC_FUSE_POOL) && pc >= 0 && net->ops[pc].fuse == 8 &&
        (o.kind == CTC_OP_CONV || o.kind == CTC_OP_MAXPOOL)) {
        const ctc_op &co = net->ops[pc].spec;
        const TensorInfo &ti = net->t[co.input], &to = net->t[pc + 1];
        pa.nimg = nimg; pa.Cs = ti.cs; pa.N = co.c_out;
        pa.H = ti.h; pa.W = ti.w; pa.P = to.h; pa.Q = to.w;
        pa.R = co.k; pa.S = co.k; pa.stride = co.stride; pa.pad = co.pad;
        pa.pool = 2;
        conv_pool = conv_pool_ok(dt, pa);
    }
    if (conv_pool) {
        s = conv_kernel_name(dt, pa);
    } else if (stem_pool) {
        const OpPlan &c = net->ops[o.kind == CTC_OP_CONV ? i : i - 1];
        ConvArgs a{};
        a.N = c.spec.c_out;
        s = stem_pool_kernel_name(a);
    } else if (o.kind == CTC_OP_CONV) {
        const TensorInfo &ti = net->t[o.input];
        const TensorInfo &to = net->t[i + 1];
        ConvArgs a{};
        a.nimg = nimg; a.Cs = ti.cs; a.N = o.c_out;
        a.H = ti.h; a.W = ti.w; a.P = to.h; a.Q = to.w;
        a.R = o.k; a.S = o.k; a.stride = o.stride; a.pad = o.pad;
        int head = -1;                      // fused IR block containing op i
        for (int h = i; h >= 0 && h >= i - 2; h--)
            if (net->ops[h].fuse == 3) { head = h; break; }
        int dpw = -1;                       // fused depthwise + pointwise pair
        for (int h = i; h >= 0 && h >= i - 1; h--)
            if (net->ops[h].fuse == 9) { dpw = h; break; }
        int bh = -1;                        // fused basic block containing op i
        for (int h = i; h >= 0 && h >= i - 1; h--)
            if (net->ops[h].fuse == 2) { bh = h; break; }
        int dh = -1;                        // fused downsampling block
        for (int h = i; h >= 0 && h >= i - 2; h--)
            if (net->ops[h].fuse == 4) { dh = h; break; }
        int sh = -1;                        // stem fused with the next block
        for (int h = i; h >= 0 && h >= i - 2; h--)
            if (net->ops[h].fuse == 5) { sh = h; break; }
        if (sh >= 0 && (net->fusion & CTC_FUSE_BLOCK) && block_fused(net, sh + 1, nimg)) {
            const TensorInfo &tb = net->t[sh + 1];
            BlockArgs b{};
            b.nimg = nimg; b.C = tb.cs; b.H = tb.h; b.W = tb.w;
            b.x0 = (const void *)1;             // naming only: with the stem
            choose_block_tile(b);
            s = block_kernel_name(b);
        } else if (dh >= 0 && (net->fusion & CTC_FUSE_BLOCK)) {
            DownArgs d{};
            d.Ci = net->t[net->ops[dh].spec.input].cs;
            s = down_kernel_name(d);
        } else if (dpw >= 0 && (net->fusion & CTC_FUSE_IR)) {
            s = "conv_dwpw";
        } else if (head >= 0 && (net->fusion & CTC_FUSE_IR)) {
            IrArgs ia{};
            ia.C = net->t[net->ops[head].spec.input].cs;
            ia.Co = net->ops[head + 2].spec.c_out;
            ia.stride = net->ops[head + 1].spec.stride;
            ia.P = net->t[head + 3].h; ia.Q = net->t[head + 3].w;
            s = ir_kernel_name(ia);
        } else if (bh >= 0 && (net->fusion & CTC_FUSE_BLOCK) && block_fused(net, bh, nimg)) {
            BlockArgs b{};
            b.nimg = nimg; b.C = a.N;
            b.head = net->ops[bh].head;
            b.H = net->t[net->ops[bh].spec.input].h;
            b.W = net->t[net->ops[bh].spec.input].w;
            choose_block_tile(b);
            s = block_kernel_name(b);
        } else if (op.dw) {
            s = dwconv_kernel_name(dt, a);
        } else {
            TileCfg tc = choose_tile(dt, a);
            s = tc.IMW > 0 ? conv_tile_name(dt, tc) : conv_kernel_name(dt, a);
        }
    } else if (o.kind == CTC_OP_MAXPOOL) {
        const TensorInfo &ti = net->t[o.input];
        const TensorInfo &to = net->t[i + 1];
        s = maxpool_kernel_name(dt, nimg, ti.h, ti.w, ti.cs, to.h, to.w, o.k,
                                o.stride);
    } else if ((o.kind == CTC_OP_GAP && i >= 2 && net->ops[i - 2].head) ||
               (o.kind == CTC_OP_FC && i >= 3 && net->ops[i - 3].head)) {
        // run by the fused block before them, when that runs fused
        const int bh = o.kind == CTC_OP_GAP ? i - 2 : i - 3;
        BlockArgs b{};
        b.nimg = nimg; b.C = net->ops[bh].spec.c_out; b.head = true;
        b.H = net->t[net->ops[bh].spec.input].h;
        b.W = net->t[net->ops[bh].spec.input].w;
        choose_block_tile(b);
        if ((net->fusion & CTC_FUSE_BLOCK) && block_fused(net, bh, nimg))
            s = block_kernel_name(b);
        else if (net->fusion & CTC_FUSE_BLOCK)
            s = "gap_fc_k<1>";
        else if (o.kind == CTC_OP_GAP)
            s = std::string("gap_k<") + tn + ">";
        else
            s = fc_name(i);
    } else if ((o.kind == CTC_OP_GAP && op.fuse == 6 && (net->fusion & CTC_FUSE_BLOCK)) ||
               (o.kind == CTC_OP_FC && i > 0 && net->ops[i - 1].fuse == 6 &&
                (net->fusion & CTC_FUSE_BLOCK))) {
        s = "gap_fc_k<1>";
    } else if (o.kind == CTC_OP_GAP) {
        s = std::string("gap_k<") + tn + ">";
    } else {
        s = fc_name(i);
    }
    snprintf(name, cap, "%s", s.c_str());
    return CTC_OK;
}

ctc_status ctc_net_fault_sites(const ctc_net *net, int32_t with_acts,
                               ctc_site_info *out, int32_t cap, int32_t *n) {
    if (!net || !n || cap < 0 || (cap > 0 && !out))
        return fail(CTC_ERR_ARG, "bad fault_sites arguments");
    if (!net->bound) return fail(CTC_ERR_STATE, "net not bound");
    std::vector<ctc_site_info> v;
    const int nops = (int)net->ops.size();
    for (int i = 0; i < nops; i++) {
        const OpPlan &o = net->ops[i];
        const std::pair<int, const std::vector<float> *> ps[] = {
            {CTC_SITE_WEIGHT, &o.w}, {CTC_SITE_BIAS, &o.b},
            {CTC_SITE_BN_MEAN, &o.mean}, {CTC_SITE_BN_VAR, &o.var},
            {CTC_SITE_BN_GAMMA, &o.gamma}, {CTC_SITE_BN_BETA, &o.beta}};
        for (const auto &p : ps) {
            if (p.second->empty()) continue;
            ctc_site_info si{};
            si.site = p.first;
            si.layer = i;
            si.elements = (int64_t)p.second->size();
            si.bits = (p.first == CTC_SITE_WEIGHT && net->dt == DT_F16) ? 16 : 32;
            v.push_back(si);
        }
    }
    if (with_acts) {
        for (int t = 0; t <= nops; t++) {
            ctc_site_info si{};
            si.site = CTC_SITE_ACT;
            si.layer = t;
            if (t == nops) {
                si.elements = net->out_cols;
                si.bits = 32;
            } else {
                const TensorInfo &ti = net->t[t];
                si.elements = (int64_t)ti.c * ti.h * ti.w;
                si.bits = ti.dt == DT_F16 ? 16 : 32;
            }
            v.push_back(si);
        }
    }
    *n = (int32_t)v.size();
    for (int i = 0; i < cap && i < (int)v.size(); i++) out[i] = v[i];
    return CTC_OK;
}

ctc_status ctc_net_set_fusion(ctc_net *net, int32_t kinds) {
    if (!net) return fail(CTC_ERR_ARG, "NULL net");
    if (kinds & ~(CTC_FUSE_IR | CTC_FUSE_BLOCK | CTC_FUSE_STEM | CTC_FUSE_POOL))
        return fail(CTC_ERR_ARG, "unknown fusion kinds 0x%x", (unsigned)kinds);
    net->fusion = kinds;
    return CTC_OK;
}

int32_t ctc_net_role(const ctc_net *net, int32_t i) {
    if (!net || i < 0 || i >= (int)net->ops.size()) return -1;
    return net->ops[i].role;
}

void ctc_net_destroy(ctc_net *net) { delete net; }

}  // extern "C"
