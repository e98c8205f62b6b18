// C ABI of the NITRO-D HIP library: argument validation, state layout, and the enqueueing of
// the kernels that make up one block's forward pass, one block's local training, the output
// layer, IntegerSGD and a whole training iteration (section 3.3).
#include <string.h>

#include <mutex>
#include <utility>
#include <vector>

#include "nitro_internal.h"
#include "probe.h"

using namespace nitro;

namespace nitro {
thread_local LaunchTimer *g_timer = nullptr;
}

// Scratch of nitro_block_forward_noalloc: a library-owned device array, one copy per device for
// the life of the process. Host code never passes the array's name to a kernel or a copy (on the
// host it is only a stand-in for the symbol): it uses the device address that
// hipGetSymbolAddress returns, looked up once per device (with that device current) by
// nitro_create.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[MAX_DEVICES] = {};

// The device address of `scratch` on `device` (which must be current); nullptr if the lookup
// fails.
void *scratch_address(int device)
{
    if (device < 0 || device >= MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess && p)
            g_scratch_ptr[device] = p;
        else
            (void)hipGetLastError();
    }
    return g_scratch_ptr[device];
}
}  // namespace

struct nitro_ctx : public LaunchTimer {
    int device = 0;
    hipStream_t stream = nullptr;
    int conv_tile = 0;                          // nitro_set_conv_tile
    int conv_persist = 0;                       // nitro_set_conv_persistent
    int aux_use = 3;                            // nitro_set_aux_streams (<= NAUX)
    uint32_t *flags = nullptr;                  // device: sticky status bits
    // streams of their own for the blocks' local training in a training iteration (the blocks'
    // backward passes depend only on their own forward state), created on first use. Only
    // NAUX of them: streams share the process's few hardware queues round-robin (4 by
    // default), and two streams on one queue run one after the other.
    static constexpr int NAUX = 3;
    hipStream_t aux[NAUX] = {};
    hipEvent_t fev[NITRO_MAX_BLOCKS] = {}, join[NAUX] = {};   // block b's forward done; aux done
    bool aux_ready = false;
    // the captured training iterations of nitro_train_step_graph, one per distinct set of
    // arguments and settings (its key), at most GCACHE; a new set replaces the least recently
    // replayed
    static constexpr int GCACHE = 16;
    struct GraphEntry {
        hipGraphExec_t exec = nullptr;
        std::vector<uint8_t> key;
        uint64_t last = 0;
    };
    GraphEntry graphs[GCACHE];
    uint64_t gclock = 0;
    // (a replay still in flight on the stream finishes before its graph is released)
    void drop_graphs()
    {
        bool any = false;
        for (auto &g : graphs) any |= g.exec != nullptr;
        if (any) (void)hipStreamSynchronize(stream);
        for (auto &g : graphs) {
            if (g.exec) (void)hipGraphExecDestroy(g.exec);
            g.exec = nullptr;
            g.key.clear();
        }
    }
    // per-kernel timing: TS_CAP slots per class in tsbuf (allocated when timing is first
    // enabled); used[c] slots of class c assigned since the last reset. A graph captured with
    // timing keeps writing its slots on every replay (ts_graph).
    static constexpr int TS_CAP = 1024;
    bool timing = false, ts_graph = false;
    uint64_t *tsbuf = nullptr;
    size_t used[TIMED_CLASSES] = {0, 0, 0};

    uint64_t *slot(int cls) override
    {
        if (by_events || !tsbuf || used[cls] >= (size_t)TS_CAP) return nullptr;
        return tsbuf + ((size_t)cls * TS_CAP + used[cls]++) * TS_WORDS;
    }
    // event timing: a pair of events per eager launch of a timed class (not inside a capture)
    bool by_events = false;
    std::vector<hipEvent_t> evpool[TIMED_CLASSES];
    size_t evused[TIMED_CLASSES] = {0, 0, 0};
    static bool capturing(hipStream_t s)
    {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        return hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
    }
    hipEvent_t next_event(int cls)
    {
        if (evused[cls] >= 2 * (size_t)TS_CAP) return nullptr;
        if (evused[cls] == evpool[cls].size()) {
            hipEvent_t e = nullptr;
            if (hipEventCreate(&e) != hipSuccess) return nullptr;
            evpool[cls].push_back(e);
        }
        return evpool[cls][evused[cls]++];
    }
    void ev_begin(int cls, hipStream_t s) override
    {
        if (!by_events || capturing(s) || evused[cls] % 2 != 0) return;
        hipEvent_t e = next_event(cls);
        if (e) (void)hipEventRecord(e, s);
    }
    void ev_end(int cls, hipStream_t s) override
    {
        if (!by_events || evused[cls] % 2 != 1) return;
        hipEvent_t e = next_event(cls);
        if (e) (void)hipEventRecord(e, s);
    }
    void drop_events()
    {
        for (auto &v : evpool) {
            for (hipEvent_t e : v) (void)hipEventDestroy(e);
            v.clear();
        }
        for (auto &u : evused) u = 0;
    }
    nitro_status ensure_aux()
    {
        if (aux_ready) return NITRO_OK;
        for (int b = 0; b < NITRO_MAX_BLOCKS; b++)
            if (hipEventCreateWithFlags(&fev[b], hipEventDisableTiming) != hipSuccess) return NITRO_EHIP;
        for (int b = 0; b < NAUX; b++) {
            if (hipStreamCreateWithFlags(&aux[b], hipStreamNonBlocking) != hipSuccess) return NITRO_EHIP;
            if (hipEventCreateWithFlags(&join[b], hipEventDisableTiming) != hipSuccess) return NITRO_EHIP;
        }
        aux_ready = true;
        return NITRO_OK;
    }
};

namespace {

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceGuard()
    {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

nitro_status hip_status()
{
    return hipGetLastError() == hipSuccess ? NITRO_OK : NITRO_EHIP;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Installs the context's launch timer for the duration of an API call.
struct TimerScope {
    LaunchTimer *prev;
    explicit TimerScope(nitro_ctx *ctx) : prev(g_timer)
    {
        g_timer = (ctx->timing || ctx->by_events) ? ctx : nullptr;
    }
    ~TimerScope() { g_timer = prev; }
};

// ------------------------------------------------------------------------------------------
// Per-layer shapes of a block.
struct LayerGeom {
    bool conv;
    ConvShape sh;             // conv: input NHWC and c_out; linear: n, c = in, co = out, h=w=1
    int64_t in_elems;         // per batch
    int64_t out_elems;        // full resolution, per batch
    int64_t sf;               // 2^8 * fan_in
    bool pad16;               // forward on the MFMA GEMM with C_in zero-padded to 16
    bool fwd_tile;            // forward on k_conv_tile (with the padded input when pad16)
    bool dx_tile;             // input gradient on k_conv_tile (g's NHWC limb planes from dW)
    bool lin_mfma;            // linear: forward and weight gradient on the int8 MFMA GEMM
};

struct BlockGeom {
    int J;
    LayerGeom L[NITRO_MAX_LAYERS];
    int64_t out_elems;        // block output (pooled if maxpool), whole batch
    int64_t d;                // per-sample learning layer input size
    int64_t out_d;            // per-sample block output size
    int lr_kh, lr_kw;         // learning layers' pooling window (1, 1: none)
    // state buffer offsets
    size_t act[NITRO_MAX_LAYERS];
    size_t code[NITRO_MAX_LAYERS];
    size_t wf[NITRO_MAX_LAYERS];   // conv: 4 int8 limb planes of W, [co][9 ci] (ci padded: 16)
    size_t wt[NITRO_MAX_LAYERS];   // conv: 4 int8 limb planes of W, [ci][9 co]
    size_t slots;                  // max slots: |W_j| (0..3), |g_j| (4..7), |W_lr| (8), |e| (9);
                                   // slot 10 word 0: the offset form's residual count
    size_t gt;                     // weight-gradient scratch: pixel-contiguous limb planes of g
    size_t xpl;                    // weight-gradient scratch: zero-padded planes of x
    size_t xpad;                   // forward scratch: a layer input with channels padded to 16
    size_t gnl;                    // backward scratch: NHWC limb planes of g [4][P][co]
    size_t part;                   // weight-gradient scratch: split-K partial sums (int64)
    bool lr_mfma;                  // learning layer on the MFMA path
    size_t lwf, lwt, lft, lpart, lepad, let;   // its scratch
    size_t lf, lfc;                // learning-pooled block output and its window indices
    size_t yhat, e, delta, g0, g1;
    size_t g16;                    // an inner layer's gradient in the escaped 16-bit form
    size_t gres, gbias, gxq;       // the first layer's g in the offset form: residual list, bias
                                   // table, sums of x (weight gradient in the form too)
    size_t nxpad, npart, ngt, nxt; // linear layers on the MFMA GEMM: padded input rows, forward
                                   // split-K partials, the weight gradient's g^T planes and x^T
    size_t total;
};

nitro_status block_geom(const nitro_block_desc *d, BlockGeom *g)
{
    if (!d || !g) return NITRO_EINVAL;
    if (d->n < 1 || d->n_layers < 1 || d->n_layers > NITRO_MAX_LAYERS) return NITRO_EINVAL;
    if (d->alpha_inv < 2) return NITRO_EINVAL;
    if (d->round != NITRO_ROUND_FLOOR && d->round != NITRO_ROUND_TRUNC) return NITRO_EINVAL;
    if (d->n_classes < 0 || (d->maxpool != 0 && d->maxpool != 1) || d->d_lr < 0) return NITRO_EINVAL;
    const int kind = d->layer[0].kind;
    if (kind != NITRO_CONV3X3 && kind != NITRO_LINEAR) return NITRO_EINVAL;
    const bool conv = kind == NITRO_CONV3X3;
    if (conv) {
        if (d->h < 1 || d->w < 1) return NITRO_EINVAL;
        if (d->maxpool && ((d->h & 1) || (d->w & 1))) return NITRO_EINVAL;
    } else {
        if (d->h != 1 || d->w != 1 || d->maxpool) return NITRO_EINVAL;
    }
    g->J = d->n_layers;
    int c = d->layer[0].c_in;
    const int64_t hw = (int64_t)d->h * d->w;
    for (int j = 0; j < g->J; j++) {
        const nitro_layer &ly = d->layer[j];
        if (ly.kind != kind || ly.c_in < 1 || ly.c_out < 1 || ly.c_in != c) return NITRO_EINVAL;
        LayerGeom &L = g->L[j];
        L.conv = conv;
        L.sh = ConvShape{d->n, conv ? d->h : 1, conv ? d->w : 1, ly.c_in, ly.c_out};
        L.in_elems = hw * ly.c_in;
        L.out_elems = hw * ly.c_out;
        L.sf = 256 * (int64_t)(conv ? 9 * ly.c_in : ly.c_in);
        const bool pool = j == d->n_layers - 1 && d->maxpool;
        L.pad16 = L.fwd_tile = L.dx_tile = false;
        L.lin_mfma = !conv && linear_mfma_ok(d->n, ly.c_in, ly.c_out);
        if (conv) {
            ConvShape s16 = L.sh;
            if (ly.c_in < 16) s16.c = 16;
            L.fwd_tile = tile_conv_fwd_ok(s16, pool, L.sf, d->alpha_inv);
            L.pad16 = ly.c_in < 16 && (L.fwd_tile || mfma_conv_fwd_ok(s16, pool));
            if (ly.c_in < 16 && !L.pad16) L.fwd_tile = false;
            L.dx_tile = dwp_ok(L.sh) && tile_conv_dx_ok(L.sh);
        }
        c = ly.c_out;
    }
    // the elementwise kernels index activations and weights with 32-bit arithmetic
    for (int j = 0; j < g->J; j++) {
        const int64_t big = g->L[j].out_elems > g->L[j].in_elems ? g->L[j].out_elems : g->L[j].in_elems;
        if ((int64_t)d->n * big >= ((int64_t)1 << 31)) return NITRO_EUNSUPPORTED;
        if (9 * (int64_t)g->L[j].sh.c * g->L[j].sh.co >= ((int64_t)1 << 31)) return NITRO_EUNSUPPORTED;
    }
    g->d = d->maxpool ? (int64_t)(d->h / 2) * (d->w / 2) * c : hw * c;
    g->out_elems = (int64_t)d->n * g->d;
    g->out_d = g->d;
    g->lr_kh = g->lr_kw = 1;
    if (conv && d->n_classes > 0 && d->d_lr > 0) {
        const int hb = d->maxpool ? d->h / 2 : d->h, wb = d->maxpool ? d->w / 2 : d->w;
        lr_pool_window(c, hb, wb, d->d_lr, &g->lr_kh, &g->lr_kw);
        g->d = (int64_t)(hb / g->lr_kh) * (wb / g->lr_kw) * c;
    }
    const bool lrpool = g->lr_kh * g->lr_kw > 1;
    // state buffer layout
    size_t off = 0;
    int64_t gmax = 0;
    for (int j = 0; j < g->J; j++) {
        const int64_t full = (int64_t)d->n * g->L[j].out_elems;
        const bool last = j == g->J - 1;
        g->act[j] = off;
        if (!last) off = align256(off + (size_t)full);
        g->code[j] = off;
        off = align256(off + (size_t)(last ? (d->maxpool ? g->out_elems : full) : full));
        if (full > gmax) gmax = full;
    }
    int64_t xpadb = 0;
    for (int j = 0; j < g->J; j++) {
        const int64_t nw = conv ? 9 * (int64_t)d->layer[j].c_in * d->layer[j].c_out : 0;
        const int64_t nwf = g->L[j].pad16 ? 9 * 16 * (int64_t)d->layer[j].c_out
                          : g->L[j].lin_mfma ? linear_scratch(d->n, d->layer[j].c_in, d->layer[j].c_out).wf_bytes / 4
                          : nw;
        g->wf[j] = off; off = align256(off + (size_t)(4 * nwf));
        g->wt[j] = off; off = align256(off + (size_t)(4 * nw));
        if (g->L[j].pad16 && (int64_t)d->n * hw * 16 > xpadb) xpadb = (int64_t)d->n * hw * 16;
    }
    g->xpad = off; off = align256(off + (size_t)xpadb);
    g->slots = off; off = align256(off + 16 * SLOT_WORDS * 4);
    g->lr_mfma = d->n_classes > 0 && !lrpool &&
                 mfma_learning_ok(d->n, g->d, d->n_classes, d->layer[g->J - 1].c_out);
    {
        LearningScratch ls{};
        if (g->lr_mfma) ls = learning_scratch(d->n, g->d, d->n_classes);
        g->lwf = off;   off = align256(off + (size_t)ls.wf_bytes);
        g->lwt = off;   off = align256(off + (size_t)ls.wt_bytes);
        g->lft = off;   off = align256(off + (size_t)ls.ft_bytes);
        g->lpart = off; off = align256(off + (size_t)ls.part_bytes);
        g->lepad = off; off = align256(off + (size_t)ls.epad_bytes);
        g->let = off;   off = align256(off + (size_t)ls.et_bytes);
    }
    g->lf = off;  off = align256(off + (size_t)(lrpool ? d->n * g->d : 0));
    g->lfc = off; off = align256(off + (size_t)(lrpool ? d->n * g->d : 0));
    int64_t gtb = 0, xpb = 0, parts = 0, gnb = 0;
    for (int j = 0; j < g->J && conv; j++) {
        const ConvShape &sh = g->L[j].sh;
        int64_t b = 0, c = 0;
        if (g->L[j].dx_tile && 4 * (int64_t)sh.n * sh.h * sh.w * sh.co > gnb)
            gnb = 4 * (int64_t)sh.n * sh.h * sh.w * sh.co;
        if (dwp_ok(sh)) {
            b = dwp_gplane_bytes(sh);
            c = dwp_partial_count(sh);
            if (dwp_xplane_bytes(sh) > xpb) xpb = dwp_xplane_bytes(sh);
        } else if (mfma_conv_dw_ok(sh) || mfma_conv_dw_smallc_ok(sh)) {
            b = 4 * (int64_t)sh.co * dw_plane_stride(sh);
            c = dw_partial_count(sh);
        } else if (smallc_dw_ok(sh)) {
            c = smallc_dw_partial_count(sh);
        }
        if (b > gtb) gtb = b;
        if (c > parts) parts = c;
    }
    g->gt = off;  off = align256(off + (size_t)gtb);
    g->xpl = off; off = align256(off + (size_t)xpb);
    g->gnl = off; off = align256(off + (size_t)gnb);
    g->part = off; off = align256(off + (size_t)parts * 8);
    const int64_t G = d->n_classes;
    g->yhat = off;  off = align256(off + (size_t)(d->n * G) * 4);
    g->e = off;     off = align256(off + (size_t)(d->n * G) * 4);
    g->delta = off; off = align256(off + (size_t)(G > 0 ? g->out_elems : 0) * 4);
    g->g0 = off;    off = align256(off + (size_t)gmax * 4);
    g->g1 = off;    off = align256(off + (size_t)(g->J > 1 ? gmax : 0) * 4);
    // (an inner layer's g, or the last layer's as the ReLU' pass writes it for the preparation)
    const bool g16_last = conv && dwp_ok(g->L[g->J - 1].sh) && !d->maxpool;
    g->g16 = off;   off = align256(off + (size_t)(g->J > 1 || g16_last ? gmax : 0) * 2);
    {
        int64_t xp = 0, pt = 0, gt = 0, xt = 0;
        for (int j = 0; j < g->J; j++) {
            if (!g->L[j].lin_mfma) continue;
            const LinearScratch ls = linear_scratch(d->n, g->L[j].sh.c, g->L[j].sh.co);
            if (ls.xpad_bytes > xp) xp = ls.xpad_bytes;
            if (ls.part_bytes > pt) pt = ls.part_bytes;
            if (ls.gt_bytes > gt) gt = ls.gt_bytes;
            if (ls.xt_bytes > xt) xt = ls.xt_bytes;
        }

        g->nxpad = off; off = align256(off + (size_t)xp);
        g->npart = off; off = align256(off + (size_t)pt);
        g->ngt = off;   off = align256(off + (size_t)gt);
        g->nxt = off;   off = align256(off + (size_t)xt);
    }
    const bool goff = conv && g->L[0].dx_tile && dwp_ok(g->L[0].sh);
    g->gres = off;  off = align256(off + (goff ? (size_t)GOFF_CAP * 4 : 0));
    g->gbias = off; off = align256(off + (goff ? (size_t)16 * 8 * g->L[0].sh.c : 0));
    g->gxq = off;   off = align256(off + (goff && dwp_goff_ok(g->L[0].sh) ? (size_t)9 * 4 * g->L[0].sh.c : 0));
    g->total = off;
    return NITRO_OK;
}

Relu make_relu(int alpha_inv, int round)
{
    return make_relu_params(alpha_inv, nitro_host_relu_mu(alpha_inv, round), round);
}

inline uint8_t *at(void *base, size_t off) { return (uint8_t *)base + off; }

// zero_slots: clear the block's max slots first (a training iteration clears every block's
// slots once, up front, instead)
// The block's last layer takes the weight-gradient kernel over padded planes and the layer
// before it the tiled forward (not pooled, being an inner layer): that forward also writes its
// output as the last layer's x rows, and the backward only zeroes their pad rows.
static bool rows_from_forward(const BlockGeom &g)
{
    if (g.J < 2) return false;
    const LayerGeom &P = g.L[g.J - 2], &L = g.L[g.J - 1];
    return P.conv && L.conv && P.fwd_tile && dwp_ok(L.sh) && L.sh.c % 16 == 0;
}

nitro_status block_forward_impl(nitro_ctx *ctx, const nitro_block_desc *desc, const BlockGeom &g,
                                const nitro_block_params *p, const int8_t *x, int8_t *a_out,
                                void *state, bool zero_slots = true, bool prepacked = false,
                                bool x_prepadded = false, bool rows_ok = true,
                                const Dropout *drop = nullptr)
{
    hipStream_t s = ctx->stream;
    const Relu rp = make_relu(desc->alpha_inv, desc->round);
    uint32_t *slots = (uint32_t *)at(state, g.slots);
    if (zero_slots && hipMemsetAsync(slots, 0, 8 * SLOT_WORDS * 4, s) != hipSuccess) return NITRO_EHIP;
    const int8_t *cur = x;
    for (int j = 0; j < g.J; j++) {
        const LayerGeom &L = g.L[j];
        const bool last = j == g.J - 1;
        const bool pool = last && desc->maxpool;
        int8_t *out = last ? a_out : (int8_t *)at(state, g.act[j]);
        uint8_t *code = at(state, g.code[j]);
        const Div sf = make_div(L.sf, desc->round);
        if (L.conv) {
            // limb planes for this call's forward and input-gradient GEMMs, and max|W_j| (the
            // training iteration packs every block's in one launch first, prepacked)
            if (!prepacked) {
                if (!L.pad16 && pack_conv_tiled_ok(L.sh.co, L.sh.c))
                    launch_pack_conv_tiled(s, p->w[j], L.sh.co, L.sh.c, (int8_t *)at(state, g.wf[j]),
                                           (int8_t *)at(state, g.wt[j]), slots + j * SLOT_WORDS);
                else
                    launch_pack_conv_weights(s, p->w[j], L.sh.co, L.sh.c, L.pad16 ? 16 : L.sh.c,
                                             (int8_t *)at(state, g.wf[j]),
                                             (int8_t *)at(state, g.wt[j]), slots + j * SLOT_WORDS);
            }
            const int8_t *wf = (const int8_t *)at(state, g.wf[j]);
            uint32_t *wmax = slots + j * SLOT_WORDS;
            ConvShape sx = L.sh;
            const int8_t *xin = cur;
            if (L.pad16) {
                // (x_prepadded: the block's input was padded by the iteration's first launch)
                int8_t *xpad = (int8_t *)at(state, g.xpad);
                if (!(j == 0 && x_prepadded))
                    launch_pad_channels16(s, cur, L.sh.n * L.sh.h * L.sh.w, L.sh.c, xpad);
                sx.c = 16;
                xin = xpad;
            }
            const bool rows = rows_ok && j == g.J - 2 && rows_from_forward(g);
            if (L.fwd_tile)
                launch_conv_fwd_tile(s, ctx->conv_tile, ctx->conv_persist, sx, xin, wf, wmax, L.sf, desc->alpha_inv, desc->round, rp,
                                     pool, out, code, ctx->flags,
                                     rows ? (int8_t *)at(state, g.xpl) : nullptr,
                                     rows ? dwp_rows_stride(g.L[j + 1].sh) : 0);
            else if (L.pad16)
                launch_conv_fwd_mfma(s, sx, xin, wf, wmax, sf, rp, pool, out, code, ctx->flags);
            else if (mfma_conv_fwd_ok(L.sh, pool))
                launch_conv_fwd_mfma(s, L.sh, cur, (const int8_t *)at(state, g.wf[j]), slots + (j) * SLOT_WORDS,
                                     sf, rp, pool, out, code, ctx->flags);
            else if (smallc_fwd_ok(L.sh))
                launch_conv_fwd_smallc(s, L.sh, cur, p->w[j], sf, rp, pool, out, code);
            else
                launch_conv_fwd(s, L.sh, cur, p->w[j], sf, rp, pool, out, code);
        } else if (L.lin_mfma) {
            const LinearScratch ls = linear_scratch(L.sh.n, L.sh.c, L.sh.co);
            if (!prepacked)
                launch_pack_linear_weights(s, p->w[j], L.sh.co, L.sh.c, ls.cip, (int8_t *)at(state, g.wf[j]),
                                           slots + j * SLOT_WORDS);
            launch_linear_fwd_mfma(s, L.sh.n, L.sh.c, L.sh.co, cur, (int8_t *)at(state, g.nxpad),
                                   (const int8_t *)at(state, g.wf[j]), slots + j * SLOT_WORDS, sf, rp, out,
                                   code, (int64_t *)at(state, g.npart), ctx->flags);
        } else {
            launch_linear_fwd_relu(s, L.sh.n, L.sh.c, L.sh.co, cur, p->w[j], sf, rp, out, code);
        }
        cur = out;
    }
    // dropout of the block output (training iterations): zeroes and "saturated" region codes
    if (drop && drop->threshold > 0)
        launch_dropout(s, a_out, at(state, g.code[g.J - 1]), g.out_elems, *drop);
    return hip_status();
}

nitro_status block_backward_impl(nitro_ctx *ctx, const nitro_block_desc *desc, const BlockGeom &g,
                                 const nitro_block_params *p, const int8_t *x, const int8_t *a_out,
                                 const int32_t *labels, const int32_t *delta_out, void *state,
                                 const nitro_block_grads *gr, const nitro_block_taps *taps,
                                 bool zero_slots = true, hipStream_t stream = nullptr,
                                 bool prepacked = false)
{
    hipStream_t s = stream ? stream : ctx->stream;
    const Relu rp = make_relu(desc->alpha_inv, desc->round);
    const int n = desc->n;
    const int G = desc->n_classes;
    const int32_t *delta = delta_out;
    int32_t *gb[2] = {(int32_t *)at(state, g.g0), (int32_t *)at(state, g.g1)};
    const int J = g.J;
    const LayerGeom &LJ = g.L[J - 1];
    uint32_t *slots = (uint32_t *)at(state, g.slots);
    // max|g_j| (4..7), max|W_lr| (8), max|e| (9) and the offset form's count (10) are produced
    // by this call
    if (zero_slots && hipMemsetAsync(slots + 4 * SLOT_WORDS, 0, 7 * SLOT_WORDS * 4, s) != hipSuccess)
        return NITRO_EHIP;
    // the offset form of g (the first layer's int64 input gradient on the tile, a block call):
    // its count is slot 10's first word; the weight gradient joins where its shape allows
    const LayerGeom &L0 = g.L[0];
    const bool goff0 = zero_slots && taps && taps->dx && L0.conv && L0.dx_tile && dwp_ok(L0.sh);
    const bool goff_dw0 = goff0 && dwp_goff_ok(L0.sh);
    const GOff go{slots + 10 * SLOT_WORDS, (uint32_t *)at(state, g.gres), (int64_t *)at(state, g.gbias),
                  goff_dw0 ? (int32_t *)at(state, g.gxq) : nullptr};
    if (goff_dw0 && hipMemsetAsync(go.xq, 0, (size_t)9 * 4 * L0.sh.c, s) != hipSuccess) return NITRO_EHIP;
    bool have_g = false;
    // The last layer's g left pooled by the learning layer and un-pooled by the weight-gradient
    // planes, which then give every other reader its values: a pooled conv block on the MFMA
    // learning layer and planes weight gradient, its input gradient (if any) on the tile, and
    // no tap asking for that g.
    const bool need_dx_last = J > 1 || (taps && taps->dx);
    const bool g_pooled = G > 0 && g.lr_mfma && desc->maxpool != 0 && LJ.conv && dwp_ok(LJ.sh) &&
                          (!need_dx_last || LJ.dx_tile) && !(taps && taps->g[J - 1]);
    if (G > 0) {
        int32_t *yhat = (int32_t *)at(state, g.yhat);
        int32_t *e = (int32_t *)at(state, g.e);

        const Div sf = make_div(256 * g.d, desc->round);
        if (g.lr_mfma) {
            LearningBuffers lb;
            lb.wf = (int8_t *)at(state, g.lwf);
            lb.wt = (int8_t *)at(state, g.lwt);
            lb.ft = (int8_t *)at(state, g.lft);
            lb.part = (int64_t *)at(state, g.lpart);
            lb.epad = (int8_t *)at(state, g.lepad);
            lb.et = (int8_t *)at(state, g.let);
            lb.wmax = slots + (8) * SLOT_WORDS;
            lb.emax = slots + (9) * SLOT_WORDS;
            lb.gmax = slots + (4 + J - 1) * SLOT_WORDS;
            launch_learning_mfma(s, n, g.d, G, a_out, p->w_lr, sf, labels, lb,
                                 at(state, g.code[J - 1]), rp, LJ.sh.h, LJ.sh.w, LJ.sh.co,
                                 desc->maxpool != 0, gb[0], taps ? taps->delta : nullptr, yhat, e,
                                 gr->dw_lr, ctx->flags, prepacked, g_pooled);
            have_g = true;
        } else if (g.lr_kh * g.lr_kw > 1) {
            // the learning layer reads the block output max-pooled to d features; its delta^fw
            // goes back through that pooling, the block's pool and NITRO-ReLU in one pass
            int32_t *dl = (int32_t *)at(state, g.delta);
            int8_t *f = (int8_t *)at(state, g.lf);
            uint8_t *fc = at(state, g.lfc);
            LrPool lp{n, desc->maxpool ? LJ.sh.h / 2 : LJ.sh.h, desc->maxpool ? LJ.sh.w / 2 : LJ.sh.w,
                      LJ.sh.co, g.lr_kh, g.lr_kw};
            launch_lr_pool(s, lp, a_out, f, fc);
            launch_linear_fwd_loss(s, n, (int)g.d, G, f, p->w_lr, sf, labels, yhat, e, ctx->flags);
            launch_linear_dw(s, n, (int)g.d, G, e, f, gr->dw_lr);
            launch_linear_dx(s, n, (int)g.d, G, e, p->w_lr, nullptr, rp, dl, nullptr, ctx->flags);
            if (taps && taps->delta)
                (void)hipMemcpyAsync(taps->delta, dl, (size_t)n * g.d * 4, hipMemcpyDeviceToDevice, s);
            launch_lr_unpool_relu_bwd(s, lp, desc->maxpool != 0, dl, fc, at(state, g.code[J - 1]), rp,
                                      gb[0], slots + (4 + J - 1) * SLOT_WORDS, ctx->flags);
            have_g = true;
        } else {
            int32_t *dl = (int32_t *)at(state, g.delta);
            launch_linear_fwd_loss(s, n, (int)g.d, G, a_out, p->w_lr, sf, labels, yhat, e, ctx->flags);
            launch_linear_dw(s, n, (int)g.d, G, e, a_out, gr->dw_lr);
            launch_linear_dx(s, n, (int)g.d, G, e, p->w_lr, nullptr, rp, dl, nullptr, ctx->flags);
            if (taps && taps->delta)
                (void)hipMemcpyAsync(taps->delta, dl, (size_t)g.out_elems * 4, hipMemcpyDeviceToDevice, s);
            delta = dl;
        }
        if (taps) {
            if (taps->yhat) (void)hipMemcpyAsync(taps->yhat, yhat, (size_t)n * G * 4, hipMemcpyDeviceToDevice, s);
            if (taps->e) (void)hipMemcpyAsync(taps->e, e, (size_t)n * G * 4, hipMemcpyDeviceToDevice, s);
        }
    }
    // g_j in the escaped 16-bit form (int16 at g16, the escapes in gb[cur]) when the layer above
    // (or, for the last layer, the ReLU' pass) wrote it so
    const int16_t *gj16 = nullptr;
    if (!have_g) {
        // the last layer's g in 16 bits where its only reader is the weight-gradient preparation
        // (no tap of it, the planes weight gradient, its input gradient (if any) on the tile)
        int16_t *g16 = nullptr;
        if (LJ.conv && !desc->maxpool && dwp_ok(LJ.sh) && (!need_dx_last || LJ.dx_tile) &&
            !(taps && taps->g[J - 1]))
            g16 = (int16_t *)at(state, g.g16);
        launch_unpool_relu_bwd(s, n, LJ.sh.h, LJ.sh.w, LJ.sh.co, desc->maxpool != 0, delta,
                               at(state, g.code[J - 1]), rp, gb[0], slots + (4 + J - 1) * SLOT_WORDS, ctx->flags,
                               g16);
        gj16 = g16;
    }
    int cur = 0;
    for (int j = J - 1; j >= 0; j--) {
        const LayerGeom &L = g.L[j];
        const int8_t *xin = j == 0 ? x : (const int8_t *)at(state, g.act[j - 1]);
        const int32_t *gj = gb[cur];
        const bool goff = j == 0 && goff0;
        if (L.conv) {
            const bool need_dx = j > 0 || (taps && taps->dx);
            if (dwp_ok(L.sh))
                launch_conv_dw_planes(s, L.sh, gj, slots + (4 + j) * SLOT_WORDS, xin,
                                      (int8_t *)at(state, g.gt), (int8_t *)at(state, g.xpl),
                                      L.dx_tile && need_dx ? (int8_t *)at(state, g.gnl) : nullptr,
                                      (int64_t *)at(state, g.part), gr->dw[j], ctx->flags,
                                      j == J - 1 && rows_from_forward(g),
                                      j == J - 1 && g_pooled ? at(state, g.code[J - 1]) : nullptr,
                                      gj16, goff ? &go : nullptr);
            else if (mfma_conv_dw_ok(L.sh) || mfma_conv_dw_smallc_ok(L.sh))
                launch_conv_dw_mfma(s, L.sh, gj, slots + (4 + j) * SLOT_WORDS, xin, (int8_t *)at(state, g.gt),
                                    (int64_t *)at(state, g.part), gr->dw[j], ctx->flags);
            else if (smallc_dw_ok(L.sh))
                launch_conv_dw_smallc(s, L.sh, gj, xin, (int64_t *)at(state, g.part), gr->dw[j]);
            else
                launch_conv_dw(s, L.sh, gj, xin, gr->dw[j]);
        } else if (L.lin_mfma) {
            launch_linear_dw_mfma(s, n, L.sh.c, L.sh.co, gj, slots + (4 + j) * SLOT_WORDS, xin,
                                  (int8_t *)at(state, g.ngt), (int8_t *)at(state, g.nxt), gr->dw[j],
                                  ctx->flags);
        } else {
            launch_linear_dw(s, n, L.sh.c, L.sh.co, gj, xin, gr->dw[j]);
        }
        if (taps && taps->g[j])
            (void)hipMemcpyAsync(taps->g[j], gj, (size_t)n * L.out_elems * 4, hipMemcpyDeviceToDevice, s);
        int32_t *dst = nullptr;
        int64_t *dst64 = nullptr;
        const uint8_t *code = nullptr;
        if (j > 0) {
            dst = gb[cur ^ 1];
            code = at(state, g.code[j - 1]);
        } else if (taps && taps->dx) {
            dst64 = taps->dx;
        }
        int16_t *dst16 = nullptr;
        if (dst && L.conv && L.dx_tile) {
            // g_{j-1} in 16 bits (with escapes) where its only reader is the weight-gradient
            // preparation of layer j-1: no tap of it, the planes weight gradient, and that
            // layer's own input gradient (if any) on the tile, which reads the prepared planes
            const LayerGeom &Lp = g.L[j - 1];
            const bool need_dx_prev = j - 1 > 0 || (taps && taps->dx);
            if (Lp.conv && dwp_ok(Lp.sh) && (!need_dx_prev || Lp.dx_tile) && !(taps && taps->g[j - 1]))
                dst16 = (int16_t *)at(state, g.g16);
        }
        if (dst || dst64) {
            uint32_t *gmax_out = j > 0 ? slots + (4 + j - 1) * SLOT_WORDS : nullptr;
            if (L.conv) {
                if (L.dx_tile) {
                    if (goff)
                        launch_goff_bias(s, (const int8_t *)at(state, g.wt[j]), L.sh.co, L.sh.c,
                                         slots + (4 + j) * SLOT_WORDS, go.bias);
                    launch_conv_dx_tile(s, ctx->conv_tile, ctx->conv_persist, L.sh, (const int8_t *)at(state, g.gnl),
                                        slots + (4 + j) * SLOT_WORDS,
                                        (const int8_t *)at(state, g.wt[j]), slots + j * SLOT_WORDS,
                                        code, rp, dst, dst64, gmax_out, ctx->flags, dst16,
                                        goff ? &go : nullptr);
                    if (goff) launch_goff_fix(s, L.sh, go, p->w[j], dst64, xin, goff_dw0 ? gr->dw[j] : nullptr);
                } else if (mfma_conv_dx_ok(L.sh))
                    launch_conv_dx_mfma(s, L.sh, gj, slots + (4 + j) * SLOT_WORDS, (const int8_t *)at(state, g.wt[j]),
                                        slots + (j) * SLOT_WORDS, code, rp, dst, dst64, gmax_out, ctx->flags);
                else
                    launch_conv_dx(s, L.sh, gj, p->w[j], code, rp, dst, dst64, gmax_out, ctx->flags);
            } else {
                launch_linear_dx(s, n, L.sh.c, L.sh.co, gj, p->w[j], code, rp, dst, dst64,
                                 ctx->flags);
            }
        }
        gj16 = dst16;
        cur ^= 1;
    }
    return hip_status();
}

bool mul_ok(int64_t a, int64_t b, int64_t *out)
{
    return !__builtin_mul_overflow(a, b, out);
}

// One IntegerSGD update as an entry of a batched launch (validation as sgd_impl). A full batch
// is launched first: its entries' gradients are complete when later entries are added.
nitro_status sgd_entry(nitro_ctx *ctx, SgdBatch &b, int32_t *w, const int64_t *dw, int64_t count,
                       int64_t gamma_inv, int64_t lambda_inv, int64_t eta_override, int32_t round,
                       hipStream_t stream = nullptr)
{
    if (!w || !dw || count < 0 || gamma_inv < 1 || lambda_inv < 0) return NITRO_EINVAL;
    if (b.n == SGD_MAX) {
        launch_sgd_batch(stream ? stream : ctx->stream, b);
        b.n = 0;
    }
    int64_t eta = eta_override;
    if (eta < 0 && !mul_ok(gamma_inv, lambda_inv, &eta)) return NITRO_EINVAL;
    SgdTensor &t = b.t[b.n++];
    t.w = w;
    t.dw = dw;
    t.count = count;
    t.gamma = make_div(gamma_inv, round);
    t.eta = make_div(eta > 0 ? eta : 1, round);
    t.decay = eta != 0;
    return NITRO_OK;
}

nitro_status sgd_impl(nitro_ctx *ctx, int32_t *w, const int64_t *dw, int64_t count,
                      int64_t gamma_inv, int64_t lambda_inv, int64_t eta_override, int32_t round)
{
    if (!w || !dw || count < 0 || gamma_inv < 1 || lambda_inv < 0) return NITRO_EINVAL;
    if (round != NITRO_ROUND_FLOOR && round != NITRO_ROUND_TRUNC) return NITRO_EINVAL;
    int64_t eta = eta_override;
    if (eta < 0 && !mul_ok(gamma_inv, lambda_inv, &eta)) return NITRO_EINVAL;
    const Div dg = make_div(gamma_inv, round);
    const Div de = make_div(eta > 0 ? eta : 1, round);
    launch_sgd(ctx->stream, w, dw, count, dg, de, eta != 0, ctx->flags);
    return hip_status();
}

// The IntegerSGD rates of an iteration: gamma^fw = AF * gamma (Eq. 6) with AF = hp->af or 2^6 G,
// eta = gamma * lambda unless given (Alg. 1). G is the learning layers' class count (or
// hp->af_classes for a block without learning layer).
struct Rates {
    int64_t gamma_fw, eta_fw, eta_lr;
};

nitro_status resolve_rates(const nitro_hparams *hp, int G, Rates *r)
{
    if (!hp || hp->gamma_inv < 1 || hp->lambda_inv_fw < 0 || hp->lambda_inv_lr < 0 || hp->af < 0 ||
        hp->af_classes < 0 || hp->reserved != 0 || hp->dropout_conv_ppm < 0 ||
        hp->dropout_conv_ppm > 1000000 || hp->dropout_lin_ppm < 0 || hp->dropout_lin_ppm > 1000000)
        return NITRO_EINVAL;
    const int64_t g = G > 0 ? G : hp->af_classes;
    const int64_t af = hp->af ? hp->af : 64 * g;
    if (af < 1) return NITRO_EINVAL;
    if (!mul_ok(af, hp->gamma_inv, &r->gamma_fw)) return NITRO_EINVAL;
    r->eta_fw = hp->eta_fw;
    r->eta_lr = hp->eta_lr;
    if (r->eta_fw < 0 && !mul_ok(r->gamma_fw, hp->lambda_inv_fw, &r->eta_fw)) return NITRO_EINVAL;
    if (r->eta_lr < 0 && !mul_ok(hp->gamma_inv, hp->lambda_inv_lr, &r->eta_lr)) return NITRO_EINVAL;
    return NITRO_OK;
}

// ------------------------------------------------------------------------------------------
// Network workspace layout.
struct NetGeom {
    BlockGeom b[NITRO_MAX_BLOCKS];
    size_t state[NITRO_MAX_BLOCKS], aout[NITRO_MAX_BLOCKS];
    size_t dw[NITRO_MAX_BLOCKS][NITRO_MAX_LAYERS], dwlr[NITRO_MAX_BLOCKS];
    size_t hyhat, he, hdw;
    int64_t hd;            // head input size
    size_t total;
};

int64_t weight_count(const nitro_layer &ly)
{
    return ly.kind == NITRO_CONV3X3 ? (int64_t)ly.c_out * 9 * ly.c_in : (int64_t)ly.c_out * ly.c_in;
}

nitro_status net_geom(const nitro_net_desc *net, NetGeom *g)
{
    if (!net || !g) return NITRO_EINVAL;
    if (net->n_blocks < 1) return NITRO_EINVAL;
    if (net->n_blocks > NITRO_MAX_BLOCKS) return NITRO_EUNSUPPORTED;
    if (net->head != 0 && net->head != 1) return NITRO_EINVAL;
    const int G = net->block[0].n_classes;
    if (G < 1) return NITRO_EINVAL;
    size_t off = 0;
    for (int b = 0; b < net->n_blocks; b++) {
        const nitro_block_desc &d = net->block[b];
        nitro_status st = block_geom(&d, &g->b[b]);
        if (st != NITRO_OK) return st;
        if (d.n_classes != G || d.n != net->block[0].n || d.alpha_inv != net->block[0].alpha_inv ||
            d.round != net->block[0].round)
            return NITRO_EINVAL;
        if (b > 0) {
            const nitro_block_desc &pd = net->block[b - 1];
            const nitro_layer &pl = pd.layer[pd.n_layers - 1];
            const bool pconv = pl.kind == NITRO_CONV3X3;
            const bool conv = d.layer[0].kind == NITRO_CONV3X3;
            if (!pconv && conv) return NITRO_EINVAL;
            if (conv) {
                const int ph = pd.maxpool ? pd.h / 2 : pd.h, pw = pd.maxpool ? pd.w / 2 : pd.w;
                if (d.h != ph || d.w != pw || d.layer[0].c_in != pl.c_out) return NITRO_EINVAL;
            } else if (pconv) {
                // a linear block reads the conv block output flattened in (h, w, c) order
                const int64_t ph = pd.maxpool ? pd.h / 2 : pd.h, pw = pd.maxpool ? pd.w / 2 : pd.w;
                if ((int64_t)d.layer[0].c_in != ph * pw * pl.c_out) return NITRO_EINVAL;
            } else if (d.layer[0].c_in != pl.c_out) {
                return NITRO_EINVAL;
            }
        }
        g->state[b] = off; off = align256(off + g->b[b].total);
        g->aout[b] = off;  off = align256(off + (size_t)g->b[b].out_elems);
        for (int j = 0; j < d.n_layers; j++) {
            g->dw[b][j] = off;
            off = align256(off + (size_t)weight_count(d.layer[j]) * 8);
        }
        g->dwlr[b] = off; off = align256(off + (size_t)G * g->b[b].d * 8);
    }
    const int L = net->n_blocks - 1;
    const int n = net->block[0].n;
    g->hd = g->b[L].out_d;
    g->hyhat = off; off = align256(off + (size_t)(net->head ? n * G : 0) * 4);
    g->he = off;    off = align256(off + (size_t)(net->head ? n * G : 0) * 4);
    g->hdw = off;   off = align256(off + (size_t)(net->head ? G * g->hd : 0) * 8);
    g->total = off;
    return NITRO_OK;
}

}  // namespace

// ============================================================================================
extern "C" {

const char *nitro_status_str(nitro_status s)
{
    switch (s) {
    case NITRO_OK: return "ok";
    case NITRO_EINVAL: return "invalid argument";
    case NITRO_EOVERFLOW: return "integer overflow: a value does not fit its declared type";
    case NITRO_ELABEL: return "label outside [0, G)";
    case NITRO_EHIP: return "HIP runtime error";
    case NITRO_ENOMEM: return "out of device memory";
    case NITRO_EUNSUPPORTED: return "unsupported by the library";
    }
    return "unknown status";
}

int64_t nitro_host_div(int64_t n, int64_t d, int32_t round)
{
    if (d < 1) return 0;
    return idiv(n, make_div(d, round));
}

int32_t nitro_host_relu_mu(int32_t alpha_inv, int32_t round)
{
    if (alpha_inv < 1) return 0;
    const int64_t s1 = idiv(-127, make_div(alpha_inv, round));
    const int64_t s2 = idiv(-127, make_div(2 * (int64_t)alpha_inv, round));
    return (int32_t)idiv(s1 + s2 + 63 + 127, make_div(4, round));
}

int32_t nitro_host_kaiming_bound(int64_t fan_in)
{
    if (fan_in < 1) return 0;
    // integer square root by bisection: the largest r with r * r <= fan_in
    int64_t lo = 1, hi = 3037000499;               // floor(sqrt(2^63 - 1))
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo + 1) / 2;
        if (mid <= fan_in / mid) lo = mid; else hi = mid - 1;
    }
    return (int32_t)((128 * 1732) / (lo * 1000));
}

nitro_status nitro_create(nitro_ctx **out, int device, void *hip_stream)
{
    if (!out) return NITRO_EINVAL;
    *out = nullptr;
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device < 0 || device >= count) return NITRO_EINVAL;
    DeviceGuard guard(device);
    nitro_ctx *c = new nitro_ctx();
    c->device = device;
    c->stream = (hipStream_t)hip_stream;
    if (hipMalloc((void **)&c->flags, 256) != hipSuccess) { delete c; return NITRO_ENOMEM; }
    if (hipMemset(c->flags, 0, 256) != hipSuccess) { (void)hipFree(c->flags); delete c; return NITRO_EHIP; }
    // the device address of the no-allocation scratch, looked up once per device (a failed
    // lookup only disables nitro_block_forward_noalloc, which then returns NITRO_EHIP)
    (void)scratch_address(device);
    *out = c;
    return NITRO_OK;
}

void nitro_destroy(nitro_ctx *ctx)
{
    if (!ctx) return;
    DeviceGuard guard(ctx->device);
    (void)hipStreamSynchronize(ctx->stream);
    ctx->drop_graphs();
    ctx->drop_events();
    if (ctx->tsbuf) (void)hipFree(ctx->tsbuf);
    if (ctx->aux_ready) {
        for (int b = 0; b < nitro_ctx::NAUX; b++) {
            (void)hipStreamSynchronize(ctx->aux[b]);
            (void)hipStreamDestroy(ctx->aux[b]);
            (void)hipEventDestroy(ctx->join[b]);
        }
        for (int b = 0; b < NITRO_MAX_BLOCKS; b++) (void)hipEventDestroy(ctx->fev[b]);
    }
    (void)hipFree(ctx->flags);
    delete ctx;
}

nitro_status nitro_set_stream(nitro_ctx *ctx, void *hip_stream)
{
    if (!ctx) return NITRO_EINVAL;
    ctx->stream = (hipStream_t)hip_stream;
    return NITRO_OK;
}

nitro_status nitro_set_conv_tile(nitro_ctx *ctx, int32_t pixels)
{
    if (!ctx || (pixels != 0 && pixels != 128 && pixels != 256)) return NITRO_EINVAL;
    ctx->conv_tile = pixels;
    return NITRO_OK;
}

nitro_status nitro_set_conv_persistent(nitro_ctx *ctx, int32_t mode)
{
    if (!ctx || mode < -1 || mode > 1) return NITRO_EINVAL;
    ctx->conv_persist = mode;
    return NITRO_OK;
}

nitro_status nitro_set_aux_streams(nitro_ctx *ctx, int32_t n)
{
    if (!ctx || n < 0 || n > nitro_ctx::NAUX) return NITRO_EINVAL;
    ctx->aux_use = n;
    return NITRO_OK;
}

nitro_status nitro_sync_status(nitro_ctx *ctx)
{
    if (!ctx) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    if (hipStreamSynchronize(ctx->stream) != hipSuccess) return NITRO_EHIP;
    uint32_t f = 0;
    if (hipMemcpy(&f, ctx->flags, 4, hipMemcpyDeviceToHost) != hipSuccess) return NITRO_EHIP;
    if (f && hipMemset(ctx->flags, 0, 4) != hipSuccess) return NITRO_EHIP;
    if (f & FLAG_OVERFLOW) return NITRO_EOVERFLOW;
    if (f & FLAG_LABEL) return NITRO_ELABEL;
    return NITRO_OK;
}

nitro_status nitro_block_query(const nitro_block_desc *desc, size_t *state_bytes)
{
    if (!state_bytes) return NITRO_EINVAL;
    BlockGeom g;
    nitro_status st = block_geom(desc, &g);
    if (st != NITRO_OK) return st;
    *state_bytes = g.total;
    return NITRO_OK;
}

nitro_status nitro_block_saved(const nitro_block_desc *desc, void *state, int32_t j,
                               int8_t **act, uint8_t **code)
{
    if (!state || !act || !code) return NITRO_EINVAL;
    BlockGeom g;
    nitro_status st = block_geom(desc, &g);
    if (st != NITRO_OK) return st;
    if (j < 0 || j >= g.J) return NITRO_EINVAL;
    *act = j == g.J - 1 ? nullptr : (int8_t *)at(state, g.act[j]);
    *code = at(state, g.code[j]);
    return NITRO_OK;
}

nitro_status nitro_block_forward(nitro_ctx *ctx, const nitro_block_desc *desc,
                                 const nitro_block_params *params, const int8_t *x,
                                 int8_t *a_out, void *state)
{
    if (!ctx || !params || !x || !a_out || !state) return NITRO_EINVAL;
    BlockGeom g;
    nitro_status st = block_geom(desc, &g);
    if (st != NITRO_OK) return st;
    for (int j = 0; j < g.J; j++)
        if (!params->w[j]) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    TimerScope timer(ctx);
    return block_forward_impl(ctx, desc, g, params, x, a_out, state);
}

nitro_status nitro_block_forward_noalloc(nitro_ctx *ctx, const nitro_block_desc *desc,
                                         const nitro_block_params *params, const int8_t *x,
                                         int8_t *a_out)
{
    if (!params || !x || !a_out) return NITRO_EINVAL;
    BlockGeom g;
    nitro_status st = block_geom(desc, &g);
    if (st != NITRO_OK) return st;
    for (int j = 0; j < g.J; j++)
        if (!params->w[j]) return NITRO_EINVAL;
    // the forward pass uses the front of the block state (saved activations and codes, weight
    // limb planes, the channel-padded input and the max slots) and, for linear layers on the
    // MFMA GEMM, their padded rows and split-K partials, which the block state keeps among the
    // backward's scratch: here they move to just behind the max slots. The size is checked
    // before the context, so that the limit holds whatever else is wrong.
    BlockGeom gf = g;
    size_t need = align256(g.slots + 16 * SLOT_WORDS * 4);
    {
        int64_t xp = 0, pt = 0;
        for (int j = 0; j < g.J; j++) {
            if (!g.L[j].lin_mfma) continue;
            const LinearScratch ls = linear_scratch(desc->n, g.L[j].sh.c, g.L[j].sh.co);
            if (ls.xpad_bytes > xp) xp = ls.xpad_bytes;
            if (ls.part_bytes > pt) pt = ls.part_bytes;
        }
        gf.nxpad = need;
        gf.npart = align256(gf.nxpad + (size_t)xp);
        need = align256(gf.npart + (size_t)pt);
    }
    if (need > NOALLOC_SCRATCH_BYTES) return NITRO_EUNSUPPORTED;
    if (!ctx) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    void *state = scratch_address(ctx->device);
    if (!state) return NITRO_EHIP;
    TimerScope timer(ctx);
    // the max slots start at zero: cleared by a kernel (no memset node if the caller captures)
    SlotList sl{};
    sl.p[0] = (uint32_t *)at(state, gf.slots);
    sl.words = 8 * SLOT_WORDS;
    launch_zero_slots(ctx->stream, sl, 1);
    return block_forward_impl(ctx, desc, gf, params, x, a_out, state, false, false, false, false);
}

nitro_status nitro_block_backward(nitro_ctx *ctx, const nitro_block_desc *desc,
                                  const nitro_block_params *params, const int8_t *x,
                                  const int8_t *a_out, const int32_t *labels,
                                  const int32_t *delta_out, void *state,
                                  const nitro_block_grads *grads, const nitro_block_taps *taps)
{
    if (!ctx || !params || !x || !a_out || !state || !grads) return NITRO_EINVAL;
    BlockGeom g;
    nitro_status st = block_geom(desc, &g);
    if (st != NITRO_OK) return st;
    for (int j = 0; j < g.J; j++)
        if (!params->w[j] || !grads->dw[j]) return NITRO_EINVAL;
    if (desc->n_classes > 0) {
        if (!labels || !params->w_lr || !grads->dw_lr) return NITRO_EINVAL;
    } else if (!delta_out) {
        return NITRO_EINVAL;
    }
    DeviceGuard guard(ctx->device);
    TimerScope timer(ctx);
    return block_backward_impl(ctx, desc, g, params, x, a_out, labels, delta_out, state, grads, taps);
}

// The one-layer block of a layer call (no pooling, no learning layer).
static nitro_status layer_block(const nitro_layer_desc *d, nitro_block_desc *b)
{
    if (!d) return NITRO_EINVAL;
    *b = nitro_block_desc{};
    b->n = d->n;
    b->h = d->h;
    b->w = d->w;
    b->n_layers = 1;
    b->layer[0] = d->layer;
    b->alpha_inv = d->alpha_inv;
    b->round = d->round;
    return NITRO_OK;
}

nitro_status nitro_layer_query(const nitro_layer_desc *desc, size_t *state_bytes)
{
    nitro_block_desc b;
    if (layer_block(desc, &b) != NITRO_OK) return NITRO_EINVAL;
    return nitro_block_query(&b, state_bytes);
}

nitro_status nitro_layer_forward(nitro_ctx *ctx, const nitro_layer_desc *desc, const int32_t *w,
                                 const int8_t *x, int8_t *a_out, void *state)
{
    nitro_block_desc b;
    if (layer_block(desc, &b) != NITRO_OK || !w) return NITRO_EINVAL;
    nitro_block_params p{};
    p.w[0] = w;
    return nitro_block_forward(ctx, &b, &p, x, a_out, state);
}

nitro_status nitro_layer_backward(nitro_ctx *ctx, const nitro_layer_desc *desc, const int32_t *w,
                                  const int8_t *x, const int8_t *a_out, const int32_t *delta,
                                  void *state, int64_t *dw, int32_t *g, int64_t *dx)
{
    nitro_block_desc b;
    if (layer_block(desc, &b) != NITRO_OK || !w || !delta || !dw) return NITRO_EINVAL;
    nitro_block_params p{};
    p.w[0] = w;
    nitro_block_grads gr{};
    gr.dw[0] = dw;
    nitro_block_taps t{};
    t.g[0] = g;
    t.dx = dx;
    return nitro_block_backward(ctx, &b, &p, x, a_out, nullptr, delta, state, &gr,
                                g || dx ? &t : nullptr);
}

nitro_status nitro_head_backward(nitro_ctx *ctx, int32_t n, int32_t d, int32_t n_classes,
                                 const int8_t *f, const int32_t *w, const int32_t *labels,
                                 int32_t round, int64_t *dw, int32_t *yhat, int32_t *e)
{
    if (!ctx || n < 1 || d < 1 || n_classes < 1 || !f || !w || !labels || !dw || !yhat || !e)
        return NITRO_EINVAL;
    if (round != NITRO_ROUND_FLOOR && round != NITRO_ROUND_TRUNC) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    const Div sf = make_div(256 * (int64_t)d, round);
    launch_linear_fwd_loss(ctx->stream, n, d, n_classes, f, w, sf, labels, yhat, e, ctx->flags);
    launch_linear_dw(ctx->stream, n, d, n_classes, e, f, dw);
    return hip_status();
}

nitro_status nitro_integer_sgd_step(nitro_ctx *ctx, int32_t *w, const int64_t *dw, int64_t count,
                                    int64_t gamma_inv, int64_t lambda_inv, int64_t eta_override,
                                    int32_t round)
{
    if (!ctx) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    return sgd_impl(ctx, w, dw, count, gamma_inv, lambda_inv, eta_override, round);
}

nitro_status nitro_net_query(const nitro_net_desc *net, size_t *workspace_bytes)
{
    if (!workspace_bytes) return NITRO_EINVAL;
    NetGeom g;
    nitro_status st = net_geom(net, &g);
    if (st != NITRO_OK) return st;
    *workspace_bytes = g.total;
    return NITRO_OK;
}

nitro_status nitro_net_block_output(const nitro_net_desc *net, void *workspace, int32_t b,
                                    int8_t **a_out)
{
    if (!workspace || !a_out) return NITRO_EINVAL;
    NetGeom g;
    nitro_status st = net_geom(net, &g);
    if (st != NITRO_OK) return st;
    if (b < 0 || b >= net->n_blocks) return NITRO_EINVAL;
    *a_out = (int8_t *)at(workspace, g.aout[b]);
    return NITRO_OK;
}

// The start of an iteration (training or inference): every block's max slots cleared in one
// launch (with block 0's input zero-padded to 16 channels where its first layer takes it so),
// then the limb planes (and max |W|) of the tiled conv layers' and the MFMA learning layers'
// weights of every block, in one launch ahead of the forward pass.
void net_setup(nitro_ctx *ctx, const nitro_net_desc *net, const NetGeom &g,
               const nitro_net_params *params, void *workspace, const int8_t *x)
{
    {
        SlotList sl{};
        sl.words = 16 * SLOT_WORDS;
        for (int b = 0; b < net->n_blocks; b++)
            sl.p[b] = (uint32_t *)at(at(workspace, g.state[b]), g.b[b].slots);
        // (with them, block 0's input zero-padded to 16 channels where its first layer takes it so)
        Pad16Args pad{};
        const BlockGeom &b0 = g.b[0];
        if (b0.L[0].conv && b0.L[0].pad16) {
            pad.x = x;
            pad.P = b0.L[0].sh.n * b0.L[0].sh.h * b0.L[0].sh.w;
            pad.c = b0.L[0].sh.c;
            pad.xpad = (int8_t *)at(at(workspace, g.state[0]), b0.xpad);
        }
        launch_zero_slots(ctx->stream, sl, net->n_blocks, &pad);
    }
    // limb planes (and max |W|) of the tiled conv layers' and the MFMA learning layers' weights
    // of every block, in one launch ahead of the forward pass
    {
        PackList pl;
        for (int b = 0; b < net->n_blocks; b++) {
            const BlockGeom &bg = g.b[b];
            void *state = at(workspace, g.state[b]);
            uint32_t *slots = (uint32_t *)at(state, bg.slots);
            for (int j = 0; j < bg.J; j++) {
                const LayerGeom &L = bg.L[j];
                if (L.lin_mfma)
                    pl.add_conv(ctx->stream, params->w[b][j], L.sh.co, L.sh.c,
                                linear_scratch(L.sh.n, L.sh.c, L.sh.co).cip, (int8_t *)at(state, bg.wf[j]),
                                nullptr, slots + j * SLOT_WORDS, 1);
                if (!L.conv) continue;
                if (!L.pad16 && pack_conv_tiled_ok(L.sh.co, L.sh.c))
                    pl.add(ctx->stream,
                           pack_conv_args(params->w[b][j], L.sh.co, L.sh.c, (int8_t *)at(state, bg.wf[j]),
                                          (int8_t *)at(state, bg.wt[j]), slots + j * SLOT_WORDS), 9);
                else
                    pl.add_conv(ctx->stream, params->w[b][j], L.sh.co, L.sh.c, L.pad16 ? 16 : L.sh.c,
                                (int8_t *)at(state, bg.wf[j]), (int8_t *)at(state, bg.wt[j]),
                                slots + j * SLOT_WORDS);
            }
            if (net->block[b].n_classes > 0 && bg.lr_mfma) {
                const LearningScratch sc = learning_scratch(net->block[b].n, bg.d, net->block[b].n_classes);
                pl.add(ctx->stream,
                       pack_matrix_args(params->w_lr[b], net->block[b].n_classes, (int)bg.d, sc.gp,
                                        (int8_t *)at(state, bg.lwf), (int8_t *)at(state, bg.lwt),
                                        slots + 8 * SLOT_WORDS), 1);
            }
        }
        pl.flush(ctx->stream);
    }
}

nitro_status nitro_block_sgd_step(nitro_ctx *ctx, const nitro_block_desc *desc,
                                  const nitro_block_weights *weights,
                                  const nitro_block_grads *grads, const nitro_hparams *hp)
{
    if (!ctx || !weights || !grads) return NITRO_EINVAL;
    BlockGeom g;
    nitro_status st = block_geom(desc, &g);
    if (st != NITRO_OK) return st;
    Rates r;
    st = resolve_rates(hp, desc->n_classes, &r);
    if (st != NITRO_OK) return st;
    for (int j = 0; j < g.J; j++)
        if (!weights->w[j] || !grads->dw[j]) return NITRO_EINVAL;
    if (desc->n_classes > 0 && (!weights->w_lr || !grads->dw_lr)) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    SgdBatch b{};
    b.flags = ctx->flags;
    if (desc->n_classes > 0) {
        st = sgd_entry(ctx, b, weights->w_lr, grads->dw_lr, (int64_t)desc->n_classes * g.d,
                       hp->gamma_inv, hp->lambda_inv_lr, r.eta_lr, desc->round);
        if (st != NITRO_OK) return st;
    }
    for (int j = 0; j < g.J; j++) {
        st = sgd_entry(ctx, b, weights->w[j], grads->dw[j], weight_count(desc->layer[j]), r.gamma_fw,
                       hp->lambda_inv_fw, r.eta_fw, desc->round);
        if (st != NITRO_OK) return st;
    }
    launch_sgd_batch(ctx->stream, b);
    return hip_status();
}

nitro_status nitro_preprocess_query(int64_t count, size_t *workspace_bytes)
{
    if (!workspace_bytes || count < 1 || count > ((int64_t)1 << 40)) return NITRO_EINVAL;
    *workspace_bytes = preprocess_workspace(count);
    return NITRO_OK;
}

nitro_status nitro_preprocess(nitro_ctx *ctx, const uint8_t *x, int64_t count, int32_t round,
                              int8_t *out, int64_t *stats, void *workspace)
{
    if (!ctx || !x || !out || !stats || !workspace) return NITRO_EINVAL;
    if (count < 1 || count > ((int64_t)1 << 40)) return NITRO_EINVAL;
    if (round != NITRO_ROUND_FLOOR && round != NITRO_ROUND_TRUNC) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    launch_preprocess(ctx->stream, x, count, round, out, stats, workspace);
    return hip_status();
}

nitro_status nitro_net_block_view(const nitro_net_desc *net, void *workspace, int32_t b,
                                  nitro_block_view *out)
{
    if (!workspace || !out) return NITRO_EINVAL;
    NetGeom g;
    nitro_status st = net_geom(net, &g);
    if (st != NITRO_OK) return st;
    if (b < 0 || b >= net->n_blocks) return NITRO_EINVAL;
    *out = nitro_block_view{};
    const BlockGeom &bg = g.b[b];
    uint8_t *state = at(workspace, g.state[b]);
    out->a_out = (int8_t *)at(workspace, g.aout[b]);
    for (int j = 0; j < bg.J; j++) {
        out->act[j] = j == bg.J - 1 ? nullptr : (int8_t *)(state + bg.act[j]);
        out->code[j] = state + bg.code[j];
        out->dw[j] = (int64_t *)at(workspace, g.dw[b][j]);
    }
    out->yhat = (int32_t *)(state + bg.yhat);
    out->e = (int32_t *)(state + bg.e);
    out->dw_lr = (int64_t *)at(workspace, g.dwlr[b]);
    return NITRO_OK;
}

nitro_status nitro_net_head_view(const nitro_net_desc *net, void *workspace, int32_t **yhat,
                                 int32_t **e, int64_t **dw)
{
    if (!workspace || !yhat || !e || !dw) return NITRO_EINVAL;
    NetGeom g;
    nitro_status st = net_geom(net, &g);
    if (st != NITRO_OK) return st;
    if (!net->head) return NITRO_EINVAL;
    *yhat = (int32_t *)at(workspace, g.hyhat);
    *e = (int32_t *)at(workspace, g.he);
    *dw = (int64_t *)at(workspace, g.hdw);
    return NITRO_OK;
}

nitro_status nitro_train_step(nitro_ctx *ctx, const nitro_net_desc *net,
                              const nitro_net_params *params, void *workspace,
                              const int8_t *x, const int32_t *labels, const nitro_hparams *hp)
{
    if (!ctx || !params || !workspace || !x || !labels || !hp) return NITRO_EINVAL;
    NetGeom g;
    nitro_status st = net_geom(net, &g);
    if (st != NITRO_OK) return st;
    const int G = net->block[0].n_classes;
    const int round = net->block[0].round;
    Rates rates;
    st = resolve_rates(hp, G, &rates);
    if (st != NITRO_OK) return st;
    const int64_t gamma_fw = rates.gamma_fw, eta_fw = rates.eta_fw, eta_lr = rates.eta_lr;
    for (int b = 0; b < net->n_blocks; b++) {
        for (int j = 0; j < net->block[b].n_layers; j++)
            if (!params->w[b][j]) return NITRO_EINVAL;
        if (!params->w_lr[b]) return NITRO_EINVAL;
    }
    if (net->head && !params->w_head) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    TimerScope timer(ctx);
    // a captured iteration with timing clears its timing slots first (every replay measures
    // afresh); every block's max slots cleared in one launch; each block's updates enqueued
    // behind its local training, the last block's and the output layer's at the end (blocks and
    // the output layer share no weights)
    if (ctx->timing && ctx->tsbuf) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(ctx->stream, &cs) == hipSuccess && cs == hipStreamCaptureStatusActive)
            launch_ts_reset(ctx->stream, ctx->tsbuf, (int64_t)TIMED_CLASSES * nitro_ctx::TS_CAP);
    }
    net_setup(ctx, net, g, params, workspace, x);
    SgdBatch sgd{};
    sgd.flags = ctx->flags;

    // 1. forward through the blocks on the context's stream (pre-update weights). A block's
    // local training (3.) needs only its own forward state and the labels, so it is enqueued as
    // soon as its forward is: on auxiliary stream b mod the number in use, which first waits for
    // an event recorded behind the block's forward, while the context's stream goes on with the
    // next block. The last block trains on the context's stream after the output layer (2.).
    // With no auxiliary stream (nitro_set_aux_streams) everything runs on the context's stream.
    st = ctx->ensure_aux();
    if (st != NITRO_OK) return st;
    const int nuse = ctx->aux_use;
    unsigned used_aux = 0;
    // every auxiliary stream that joined the iteration is joined back to the context's stream
    // before returning, on error too: a capture can only end once every stream forked from the
    // capturing one has been joined into it
    auto join_aux = [&]() -> bool {
        bool ok = true;
        for (int a = 0; a < nuse; a++) {
            if (!(used_aux & (1u << a))) continue;
            ok &= hipEventRecord(ctx->join[a], ctx->aux[a]) == hipSuccess;
            ok &= hipStreamWaitEvent(ctx->stream, ctx->join[a], 0) == hipSuccess;
        }
        used_aux = 0;
        return ok;
    };
    auto fail = [&](nitro_status e) -> nitro_status {
        (void)join_aux();
        return e;
    };
    // IntegerSGD (Alg. 1) of block b's learning layer (gamma) and forward layers (AF gamma), on
    // the stream of the block's local training, right after it: nothing later in the iteration
    // reads these weights (the block's backward reads its packed limb planes, and no other
    // block touches them)
    auto block_sgd = [&](int b, hipStream_t bs) -> nitro_status {
        const nitro_block_desc &d = net->block[b];
        SgdBatch bb{};
        bb.flags = ctx->flags;
        nitro_status e = sgd_entry(ctx, bb, params->w_lr[b], (const int64_t *)at(workspace, g.dwlr[b]),
                                   (int64_t)G * g.b[b].d, hp->gamma_inv, hp->lambda_inv_lr, eta_lr,
                                   round, bs);
        for (int j = 0; j < d.n_layers && e == NITRO_OK; j++)
            e = sgd_entry(ctx, bb, params->w[b][j], (const int64_t *)at(workspace, g.dw[b][j]),
                          weight_count(d.layer[j]), gamma_fw, hp->lambda_inv_fw, eta_fw, round, bs);
        if (e == NITRO_OK) launch_sgd_batch(bs, bb);
        return e;
    };
    auto backward = [&](int b, hipStream_t bs) -> nitro_status {
        const nitro_block_desc &d = net->block[b];
        const int8_t *xin = b == 0 ? x : (const int8_t *)at(workspace, g.aout[b - 1]);
        nitro_block_params bp{};
        nitro_block_grads gr{};
        for (int j = 0; j < d.n_layers; j++) {
            bp.w[j] = params->w[b][j];
            gr.dw[j] = (int64_t *)at(workspace, g.dw[b][j]);
        }
        bp.w_lr = params->w_lr[b];
        gr.dw_lr = (int64_t *)at(workspace, g.dwlr[b]);
        return block_backward_impl(ctx, &d, g.b[b], &bp, xin, (const int8_t *)at(workspace, g.aout[b]),
                                   labels, nullptr, at(workspace, g.state[b]), &gr, nullptr, false,
                                   bs, true);
    };
    const int8_t *cur = x;
    for (int b = 0; b < net->n_blocks; b++) {
        nitro_block_params bp{};
        for (int j = 0; j < net->block[b].n_layers; j++) bp.w[j] = params->w[b][j];
        bp.w_lr = params->w_lr[b];
        int8_t *aout = (int8_t *)at(workspace, g.aout[b]);
        const bool bconv = net->block[b].layer[0].kind == NITRO_CONV3X3;
        const int64_t ppm = bconv ? hp->dropout_conv_ppm : hp->dropout_lin_ppm;
        Dropout drop{(uint64_t)((ppm << 32) / 1000000), hp->dropout_seed, (uint64_t)hp->dropout_step,
                     b, net->block[b].maxpool};
        st = block_forward_impl(ctx, &net->block[b], g.b[b], &bp, cur, aout, at(workspace, g.state[b]),
                                false, true, b == 0, true, &drop);
        if (st != NITRO_OK) return fail(st);
        cur = aout;
        if (b + 1 == net->n_blocks) break;
        hipStream_t bs = ctx->stream;
        if (nuse > 0) {
            const int a = b % nuse;
            bs = ctx->aux[a];
            if (hipEventRecord(ctx->fev[b], ctx->stream) != hipSuccess) return fail(NITRO_EHIP);
            used_aux |= 1u << a;
            if (hipStreamWaitEvent(bs, ctx->fev[b], 0) != hipSuccess) return fail(NITRO_EHIP);
        }
        st = backward(b, bs);
        if (st != NITRO_OK) return fail(st);
        st = block_sgd(b, bs);
        if (st != NITRO_OK) return fail(st);
    }
    // 2. output layer: global gradient (its update comes with the others, step 4)
    const int n = net->block[0].n;
    int64_t *hdw = (int64_t *)at(workspace, g.hdw);
    if (net->head) {
        const int64_t d = g.hd;
        const Div sf = make_div(256 * d, round);
        launch_linear_fwd_loss(ctx->stream, n, (int)d, G, cur, params->w_head, sf, labels,
                               (int32_t *)at(workspace, g.hyhat), (int32_t *)at(workspace, g.he),
                               ctx->flags);
        launch_linear_dw(ctx->stream, n, (int)d, G, (const int32_t *)at(workspace, g.he), cur, hdw);
    }
    // 3. the last block's local training; the context's stream then waits for the others
    st = backward(net->n_blocks - 1, ctx->stream);
    if (st != NITRO_OK) return fail(st);
    if (!join_aux()) return NITRO_EHIP;
    // 4. IntegerSGD (Alg. 1) of the output layer and of the last block (the other blocks' updates
    // were enqueued behind their local training)
    if (net->head) {
        st = sgd_entry(ctx, sgd, params->w_head, hdw, (int64_t)G * g.hd, hp->gamma_inv,
                       hp->lambda_inv_lr, eta_lr, round);
        if (st != NITRO_OK) return st;
    }
    {
        const int b = net->n_blocks - 1;
        const nitro_block_desc &d = net->block[b];
        st = sgd_entry(ctx, sgd, params->w_lr[b], (const int64_t *)at(workspace, g.dwlr[b]),
                       (int64_t)G * g.b[b].d, hp->gamma_inv, hp->lambda_inv_lr, eta_lr, round);
        if (st != NITRO_OK) return st;
        for (int j = 0; j < d.n_layers; j++) {
            st = sgd_entry(ctx, sgd, params->w[b][j], (const int64_t *)at(workspace, g.dw[b][j]),
                           weight_count(d.layer[j]), gamma_fw, hp->lambda_inv_fw, eta_fw, round);
            if (st != NITRO_OK) return st;
        }
    }
    launch_sgd_batch(ctx->stream, sgd);
    return hip_status();
}

nitro_status nitro_net_infer(nitro_ctx *ctx, const nitro_net_desc *net,
                             const nitro_net_params *params, void *workspace, const int8_t *x,
                             int32_t *yhat, int32_t *pred)
{
    if (!ctx || !params || !workspace || !x || !yhat || !pred) return NITRO_EINVAL;
    NetGeom g;
    nitro_status st = net_geom(net, &g);
    if (st != NITRO_OK) return st;
    for (int b = 0; b < net->n_blocks; b++)
        for (int j = 0; j < net->block[b].n_layers; j++)
            if (!params->w[b][j]) return NITRO_EINVAL;
    const int L = net->n_blocks - 1;
    if (net->head ? !params->w_head : !params->w_lr[L]) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    TimerScope timer(ctx);
    hipStream_t s = ctx->stream;
    const int n = net->block[0].n, G = net->block[0].n_classes;
    const int round = net->block[0].round;
    net_setup(ctx, net, g, params, workspace, x);
    const int8_t *cur = x;
    for (int b = 0; b < net->n_blocks; b++) {
        nitro_block_params bp{};
        for (int j = 0; j < net->block[b].n_layers; j++) bp.w[j] = params->w[b][j];
        int8_t *aout = (int8_t *)at(workspace, g.aout[b]);
        st = block_forward_impl(ctx, &net->block[b], g.b[b], &bp, cur, aout, at(workspace, g.state[b]),
                                false, true, b == 0);
        if (st != NITRO_OK) return st;
        cur = aout;
    }
    // the prediction: the output layer on the last block's output, or the last block's learning
    // layer (on its learning pooling, if any)
    const BlockGeom &lb = g.b[L];
    const int8_t *f = cur;
    int64_t d = net->head ? g.hd : lb.d;
    const int32_t *w = net->head ? params->w_head : params->w_lr[L];
    if (!net->head && lb.lr_kh * lb.lr_kw > 1) {
        const nitro_block_desc &ld = net->block[L];
        const LayerGeom &LJ = lb.L[lb.J - 1];
        LrPool lp{n, ld.maxpool ? LJ.sh.h / 2 : LJ.sh.h, ld.maxpool ? LJ.sh.w / 2 : LJ.sh.w, LJ.sh.co,
                  lb.lr_kh, lb.lr_kw};
        uint8_t *state = at(workspace, g.state[L]);
        launch_lr_pool(s, lp, cur, (int8_t *)(state + lb.lf), state + lb.lfc);
        f = (const int8_t *)(state + lb.lf);
    }
    launch_linear_fwd_loss(s, n, (int)d, G, f, w, make_div(256 * d, round), nullptr, yhat, nullptr,
                           ctx->flags);
    launch_argmax_rows(s, n, G, yhat, pred);
    return hip_status();
}

// The graph of this key (descriptors, parameters, buffers, hyper-parameters, the context's
// stream and settings): the one kept for it, or a new capture of one iteration.
static nitro_status graph_for_key(nitro_ctx *ctx, const nitro_net_desc *net,
                                  const nitro_net_params *params, void *workspace, const int8_t *x,
                                  const int32_t *labels, const nitro_hparams *hp,
                                  nitro_ctx::GraphEntry **out)
{
    if (!ctx || !net || !params || !workspace || !x || !labels || !hp) return NITRO_EINVAL;
    if (!ctx->stream) return NITRO_EINVAL;           // the legacy default stream cannot capture
    DeviceGuard guard(ctx->device);
    std::vector<uint8_t> key;
    auto put = [&](const void *p, size_t n) {
        const uint8_t *b = (const uint8_t *)p;
        key.insert(key.end(), b, b + n);
    };
    put(net, sizeof(*net));
    put(params, sizeof(*params));
    put(&workspace, sizeof(workspace));
    put(&x, sizeof(x));
    put(&labels, sizeof(labels));
    put(hp, sizeof(*hp));
    put(&ctx->stream, sizeof(ctx->stream));
    put(&ctx->timing, sizeof(ctx->timing));
    put(&ctx->aux_use, sizeof(ctx->aux_use));
    put(&ctx->conv_tile, sizeof(ctx->conv_tile));
    put(&ctx->conv_persist, sizeof(ctx->conv_persist));
    nitro_ctx::GraphEntry *ge = nullptr;
    for (auto &g : ctx->graphs)
        if (g.exec && g.key == key) ge = &g;
    if (!ge) {
        ge = &ctx->graphs[0];
        for (auto &g : ctx->graphs)
            if (!g.exec || (ge->exec && g.last < ge->last)) ge = &g;
        if (ge->exec) {
            if (hipStreamSynchronize(ctx->stream) != hipSuccess) return NITRO_EHIP;
            (void)hipGraphExecDestroy(ge->exec);
        }
        ge->exec = nullptr;
        ge->key.clear();
        nitro_status st = ctx->ensure_aux();
        if (st != NITRO_OK) return st;
        for (auto &u : ctx->used) u = 0;
        if (hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeRelaxed) != hipSuccess)
            return NITRO_EHIP;
        st = nitro_train_step(ctx, net, params, workspace, x, labels, hp);
        hipGraph_t graph = nullptr;
        const hipError_t e = hipStreamEndCapture(ctx->stream, &graph);
        if (st == NITRO_OK && e != hipSuccess) st = NITRO_EHIP;
        // every auxiliary stream that joined the capture must have left it with the capturing
        // stream: one still capturing was forked and not joined back, and its graph is unusable
        for (int a = 0; a < nitro_ctx::NAUX; a++)
            if (ctx->aux[a] && nitro_ctx::capturing(ctx->aux[a])) st = NITRO_EHIP;
        if (st == NITRO_OK && hipGraphInstantiate(&ge->exec, graph, nullptr, nullptr, 0) != hipSuccess) {
            ge->exec = nullptr;
            st = NITRO_EHIP;
        }
        // (a graph is handed out only by a capture that ended well; after a failed end the
        // pointer is not one to release)
        if (graph && e == hipSuccess) (void)hipGraphDestroy(graph);
        (void)hipGetLastError();
        if (st != NITRO_OK) return st;
        ge->key = std::move(key);
        ctx->ts_graph = ctx->timing && ctx->tsbuf;
    }
    ge->last = ++ctx->gclock;
    *out = ge;
    return NITRO_OK;
}

nitro_status nitro_train_step_graph(nitro_ctx *ctx, const nitro_net_desc *net,
                                    const nitro_net_params *params, void *workspace,
                                    const int8_t *x, const int32_t *labels, const nitro_hparams *hp)
{
    nitro_ctx::GraphEntry *ge = nullptr;
    const nitro_status st = graph_for_key(ctx, net, params, workspace, x, labels, hp, &ge);
    if (st != NITRO_OK) return st;
    DeviceGuard guard(ctx->device);
    if (hipGraphLaunch(ge->exec, ctx->stream) != hipSuccess) return NITRO_EHIP;
    return NITRO_OK;
}

nitro_status nitro_train_step_graph_prepare(nitro_ctx *ctx, const nitro_net_desc *net,
                                            const nitro_net_params *params, void *workspace,
                                            const int8_t *x, const int32_t *labels,
                                            const nitro_hparams *hp)
{
    nitro_ctx::GraphEntry *ge = nullptr;
    return graph_for_key(ctx, net, params, workspace, x, labels, hp, &ge);
}

nitro_status nitro_kernel_timing(nitro_ctx *ctx, int32_t enable)
{
    if (!ctx) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    if (enable < 0 || enable > 2) return NITRO_EINVAL;
    // graphs captured before hold the timing state and slot assignment of their capture
    ctx->drop_graphs();
    (void)hipStreamSynchronize(ctx->stream);
    ctx->drop_events();
    ctx->by_events = enable == 2;
    ctx->timing = enable == 1;
    if (ctx->timing) {
        const int64_t nslots = (int64_t)TIMED_CLASSES * nitro_ctx::TS_CAP;
        if (!ctx->tsbuf && hipMalloc((void **)&ctx->tsbuf, (size_t)nslots * TS_WORDS * 8) != hipSuccess) {
            ctx->tsbuf = nullptr;
            ctx->timing = false;
            return NITRO_ENOMEM;
        }
        launch_ts_reset(ctx->stream, ctx->tsbuf, nslots);
        if (hipGetLastError() != hipSuccess) return NITRO_EHIP;
    }
    for (auto &u : ctx->used) u = 0;
    ctx->ts_graph = false;
    return NITRO_OK;
}

nitro_status nitro_mfma_rate(nitro_ctx *ctx, int32_t waves_per_simd, int32_t iters, double *tops)
{
    if (!ctx || !tops || waves_per_simd < 1 || waves_per_simd > 4 || iters < 1) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, ctx->device) != hipSuccess ||
        cus < 1)
        return NITRO_EHIP;
    // 4-wave workgroups, one wave per SIMD: waves_per_simd workgroups per compute unit
    const int grid = cus * waves_per_simd;
    int32_t *out = nullptr;
    if (hipMalloc((void **)&out, (size_t)grid * 256 * sizeof(int32_t)) != hipSuccess) return NITRO_ENOMEM;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    nitro_status st = NITRO_OK;
    float ms = 0.f;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) st = NITRO_EHIP;
    if (st == NITRO_OK) {
        launch_mfma_rate(ctx->stream, grid, iters < 64 ? iters : 64, out);     // warm-up (clocks)
        if (hipEventRecord(e0, ctx->stream) != hipSuccess) st = NITRO_EHIP;
        launch_mfma_rate(ctx->stream, grid, iters, out);
        if (hipGetLastError() != hipSuccess || hipEventRecord(e1, ctx->stream) != hipSuccess ||
            hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess ||
            !(ms > 0.f))
            st = NITRO_EHIP;
    }
    if (st == NITRO_OK) *tops = (double)mfma_rate_ops(grid, iters) / (ms * 1e-3) / 1e12;
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    (void)hipFree(out);
    return st;
}

nitro_status nitro_kernel_time(nitro_ctx *ctx, int32_t cls, double *ms, int64_t *launches)
{
    if (!ctx || cls < 0 || cls >= TIMED_CLASSES || !ms || !launches) return NITRO_EINVAL;
    DeviceGuard guard(ctx->device);
    *ms = 0.0;
    *launches = 0;
    if (ctx->by_events) {
        // pairs recorded since the last read; then the pool's events are reused
        if (hipStreamSynchronize(ctx->stream) != hipSuccess) return NITRO_EHIP;
        const size_t pairs = ctx->evused[cls] / 2;
        for (size_t i = 0; i < pairs; i++) {
            float t = 0.f;
            if (hipEventSynchronize(ctx->evpool[cls][2 * i + 1]) != hipSuccess ||
                hipEventElapsedTime(&t, ctx->evpool[cls][2 * i], ctx->evpool[cls][2 * i + 1]) != hipSuccess)
                return NITRO_EHIP;
            *ms += t;
        }
        *launches = (int64_t)pairs;
        ctx->evused[cls] = 0;
        return NITRO_OK;
    }
    if (!ctx->tsbuf || ctx->used[cls] == 0) return NITRO_OK;
    if (hipStreamSynchronize(ctx->stream) != hipSuccess) return NITRO_EHIP;
    int khz = 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, ctx->device) != hipSuccess ||
        khz <= 0)
        return NITRO_EHIP;
    const size_t n = ctx->used[cls];
    std::vector<uint64_t> h(n * TS_WORDS);
    uint64_t *src = ctx->tsbuf + (size_t)cls * nitro_ctx::TS_CAP * TS_WORDS;
    if (hipMemcpy(h.data(), src, h.size() * 8, hipMemcpyDeviceToHost) != hipSuccess) return NITRO_EHIP;
    double tot = 0.0;
    int64_t cnt = 0;
    for (size_t i = 0; i < n; i++) {
        uint64_t t0 = ~(uint64_t)0, t1 = 0;
        for (int w = 0; w < TS_SPREAD; w++) {
            t0 = h[i * TS_WORDS + w] < t0 ? h[i * TS_WORDS + w] : t0;
            t1 = h[i * TS_WORDS + TS_SPREAD + w] > t1 ? h[i * TS_WORDS + TS_SPREAD + w] : t1;
        }
        if (t1 > t0) {
            tot += (double)(t1 - t0) / khz;    // ticks / (ticks per ms)
            cnt++;
        }
    }
    *ms = tot;
    *launches = cnt;
    if (!ctx->ts_graph) {
        // eager launches: the next read covers the launches after this one
        ctx->used[cls] = 0;
        launch_ts_reset(ctx->stream, src, nitro_ctx::TS_CAP);
    }
    return NITRO_OK;
}

}  // extern "C"
