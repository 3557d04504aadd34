// Host runtime of the HetPipe stage step and WSP engine: the C ABI of
// include/hetpipe.h.
//
//  * hp_stage: validates the layer list, derives every layer's shape and
//    parameter offsets, plans each contraction (tile shape, split-K), owns the
//    activation stash, per-layer gradient buffers and one shared workspace,
//    and enqueues the forward / backward launch sequence on its stream.
//    ReLUs that directly follow a conv, FC, batch-norm or residual add whose
//    only consumer they are are fused into the producer's kernel.
//  * hp_ps / hp_vw: the parameter server and the virtual workers.  Device
//    state (w_g, the weight ring, u~) is updated by the kernels in wsp.hip;
//    clocks, the push/pull protocol and the version vectors are host integers
//    updated synchronously, so bookkeeping never waits on the device.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "hetpipe.h"
#include "kernels.h"

using namespace hp;

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

#define HP_HIP(expr)                                                                  \
    do {                                                                              \
        hipError_t _e = (expr);                                                       \
        if (_e != hipSuccess)                                                         \
            return fail(_e == hipErrorOutOfMemory ? HP_ERR_NOMEM : HP_ERR_HIP,         \
                        "%s failed: %s", #expr, hipGetErrorString(_e));               \
    } while (0)

struct Node {
    hp_layer L{};
    int inH = 0, inW = 0, inC = 0;      // per-image input shape (in0)
    int H = 0, W = 0, C = 0;            // per-image output shape
    size_t out_elems = 0;               // batch * H * W * C
    int consumers = 0;
    bool relu_fused = false;            // producer applies the ReLU (this node is a ReLU)
    bool fuses_relu = false;            // this node applies its consumer ReLU
    int relu_node = -1;                 // ... which is this node
    float* y = nullptr;                 // forward output (a fused ReLU aliases its producer)
    float* g = nullptr;                 // gradient of the output
    bool g_written = false;
    // after a backward pass: the buffer holding the gradient of this value
    // (NULL where none does: see hp_stage_layer_buffers)
    const float* g_final = nullptr;
    const float* g_alias = nullptr;     // gradient handed over without a copy (ReLU -> BN, add -> sole-consumer input)
    bool g_shared = false;              // g_alias is a buffer this value's other consumers accumulate into
    bool add_share[2] = {false, false}; // (add) input 0 / 1 may take this gradient buffer as its own
    int mask_into = -1;                 // data gradient goes to this producer, ReLU-masked
    bool bias_in_wgrad = false;         // bias gradient computed by the weight-gradient GEMM
    bool bwd_by_consumer = false;       // (ReLU) its backward is fused into its consumer
    bool wgrad_side = false;            // weight gradient on the stage's second stream
    size_t p_off = 0, p_cnt = 0;        // all parameters of the node
    size_t w_off = 0, b_off = 0;        // conv/fc weight, bias; bn gamma, beta
    ConvGeo geo{};
    GemmPlan fwd{}, dgrad{}, wgrad{};
    float* mean = nullptr;
    float* invstd = nullptr;
    // bf16 mode: bf16 copy of this node's output, read by contractions that
    // stage bf16 operands directly (made once per forward pass)
    uint16_t* y16 = nullptr;
    bool y16_ready = false;
    // bf16 mode, conv / FC: bf16 copy of this node's output gradient (written by
    // the BN backward that produces it, else cast before the weight gradient)
    uint16_t* g16 = nullptr;
    bool g16_ready = false;
    // max-pool with overlapping windows: the tap of each window's first
    // maximum, recorded by the forward pass for the backward pass
    uint8_t* arg = nullptr;
    // conv whose input channel count is not a multiple of the contraction's
    // vector width (the image layer, C = 3): forward and weight gradient run
    // on copies padded with zero channels to padC (input, weights; bf16 mode:
    // their bf16 copies), the padded weight gradient is compacted into grad
    // conv whose only consumer is a batch norm: its forward contraction writes
    // per-tile column statistics (mean, squared deviations; stats_nb row
    // tiles of stats_rb rows) and the batch norm merges them
    float* stats = nullptr;
    int stats_nb = 0;
    long stats_rb = 0;
    int padC = 0;
    ConvGeo geo_p{};
    float* xp = nullptr;
    float* wp = nullptr;
    float* dwp = nullptr;
    uint16_t* xp16 = nullptr;
    uint16_t* wp16 = nullptr;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

struct StageTimer {
    bool on = false;
    // layer (node index, -1 for stage-level work) and pass (0 forward, 1
    // backward) that the next records belong to
    int node = -1, phase = 0;
    struct Rec { hipEvent_t a, b; int cat, node, phase; };
    std::vector<Rec> recs;          // recorded, not yet read
    std::vector<hipEvent_t> pool;   // free events
    hipEvent_t take() {
        if (!pool.empty()) { hipEvent_t e = pool.back(); pool.pop_back(); return e; }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
    int cur = -1;
    hipEvent_t cur_a = nullptr;
    void begin(int cat, hipStream_t s) {
        if (!on) return;
        cur_a = take();
        cur = cat;
        if (cur_a) (void)hipEventRecord(cur_a, s);
    }
    // drop the open record: the layer launched nothing of its own
    void cancel() {
        if (!on || !cur_a) return;
        pool.push_back(cur_a);
        cur_a = nullptr;
    }
    void end(hipStream_t s) {
        if (!on || !cur_a) return;
        hipEvent_t b = take();
        if (!b) return;
        (void)hipEventRecord(b, s);
        recs.push_back({cur_a, b, cur, node, phase});
        cur_a = nullptr;
    }
    ~StageTimer() {
        for (auto& r : recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
        for (auto e : pool) (void)hipEventDestroy(e);
    }
};

struct hp_stage {
    StageTimer timer;
    std::vector<Node> nodes;
    int batch = 0, H = 0, W = 0, C = 0;
    int dtype = HP_FP32;
    hipStream_t stream = nullptr;
    size_t P = 0;
    size_t ws_floats = 0;
    float* ws = nullptr;
    std::vector<void*> allocs;
    size_t bytes = 0;
    // device bytes per layer (buffers that belong to one layer's value,
    // gradient or statistics) and the stage-level rest (workspaces, weight
    // copies, the input copy); dev_alloc charges cur_node (-1: stage level)
    std::vector<size_t> node_bytes;
    size_t shared_bytes = 0;
    int cur_node = -1;
    bool has_loss = false;
    // bf16 mode with bf16 operands in memory: copies of the weights, of the
    // stage input and (scratch, one conv at a time) of a conv's output gradient
    uint16_t* w16 = nullptr;
    // transposed copies [C][R][S][K] of the weights of the convs whose data
    // gradient runs on k-major operands, and the device table that makes them
    uint16_t* w16t = nullptr;
    WtLayer* wt_table = nullptr;
    int wt_layers = 0, wt_tiles_total = 0;
    uint16_t* x16 = nullptr;
    bool x16_ready = false;
    // the weight gradients run on a second stream beside the data-gradient
    // chain (they only feed the caller's gradient vector), with a workspace
    // of their own; events order the two streams
    hipStream_t side = nullptr;
    std::vector<hipEvent_t> evs;
    size_t ev_next = 0;
    float* ws2 = nullptr;
    size_t ws2_floats = 0;
    // forward bookkeeping for backward
    const float* fwd_w = nullptr;
    const float* fwd_x = nullptr;
    bool fwd_done = false;
    // the last backward pass's input gradient (caller's dx, may be NULL)
    const float* bwd_dx = nullptr;
    int device = 0;                 // the HIP device current at creation
};

struct hp_vw;

struct hp_ps {
    StageTimer timer;
    size_t P = 0;
    float* wg = nullptr;
    int N = 0, D = 0;
    hipStream_t stream = nullptr;
    std::vector<int> clock;          // local clock of each VW
    std::vector<int64_t> pushed;     // waves of each VW contained in w_g
    std::vector<hp_vw*> vws;
    int cg = 0;
};

struct hp_vw {
    hp_ps* ps = nullptr;
    int id = 0;
    int W = 1;
    size_t P = 0, stride = 0;
    float* ring = nullptr;
    float* ut = nullptr;
    float* vel = nullptr;      // momentum velocity (allocated by hp_vw_set_momentum)
    float mu = 0.f;
    int64_t p = 0;
    int c = 0, g = 0;
    int inflight = 0;                      // started, not yet completed (at most W)
    bool push_due = false, need_pull = false;
    std::vector<std::vector<int64_t>> V;   // [W][N] version vectors of the ring slots
};

namespace {

int dev_alloc(hp_stage* st, float** p, size_t floats) {
    if (floats == 0) { *p = nullptr; return HP_OK; }
    void* q = nullptr;
    hipError_t e = hipMalloc(&q, floats * sizeof(float));
    if (e != hipSuccess)
        return fail(e == hipErrorOutOfMemory ? HP_ERR_NOMEM : HP_ERR_HIP,
                    "hipMalloc(%zu bytes): %s", floats * sizeof(float), hipGetErrorString(e));
    st->allocs.push_back(q);
    st->bytes += floats * sizeof(float);
    if (st->cur_node >= 0 && st->cur_node < (int)st->node_bytes.size())
        st->node_bytes[st->cur_node] += floats * sizeof(float);
    else
        st->shared_bytes += floats * sizeof(float);
    *p = (float*)q;
    return HP_OK;
}

int dev_alloc16(hp_stage* st, uint16_t** p, size_t n) {
    float* q = nullptr;
    int rc = dev_alloc(st, &q, (n + 1) / 2);
    *p = reinterpret_cast<uint16_t*>(q);
    return rc;
}

int num_cus() {
    int dev = 0, n = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    return n > 0 ? n : 256;
}

int shape_of(const hp_stage* st, int idx, int& H, int& W, int& C) {
    if (idx == -1) { H = st->H; W = st->W; C = st->C; return HP_OK; }
    if (idx < 0 || idx >= (int)st->nodes.size()) return HP_ERR_ARG;
    const Node& n = st->nodes[idx];
    H = n.H; W = n.W; C = n.C;
    return HP_OK;
}

int build_stage(hp_stage* st, const hp_layer* layers, int n_layers) {
    st->nodes.resize(n_layers);
    const int cus = num_cus();
    size_t off = 0;
    for (int i = 0; i < n_layers; ++i) {
        Node& nd = st->nodes[i];
        nd.L = layers[i];
        const hp_layer& L = nd.L;
        if (L.in0 < -1 || L.in0 >= i)
            return fail(HP_ERR_ARG, "layer %d: input %d is not an earlier layer", i, L.in0);
        if (L.in0 >= 0 && st->nodes[L.in0].L.kind == HP_SOFTMAX_CE)
            return fail(HP_ERR_ARG, "layer %d reads the loss head", i);
        shape_of(st, L.in0, nd.inH, nd.inW, nd.inC);
        if (L.in0 >= 0) st->nodes[L.in0].consumers++;
        const int B = st->batch;
        switch (L.kind) {
            case HP_CONV:
            case HP_FC: {
                int R = L.R, S = L.S, stride = L.stride, pad = L.pad;
                int inH = nd.inH, inW = nd.inW, inC = nd.inC;
                if (L.kind == HP_FC) {
                    // an FC layer is a 1x1 convolution over the flattened input
                    inC = nd.inH * nd.inW * nd.inC;
                    inH = inW = 1;
                    R = S = stride = 1;
                    pad = 0;
                    if (L.C != inC)
                        return fail(HP_ERR_ARG, "layer %d: FC expects %d inputs, got %d", i, L.C, inC);
                } else if (L.C != inC) {
                    return fail(HP_ERR_ARG, "layer %d: conv expects %d channels, got %d", i, L.C, inC);
                }
                if (L.K <= 0 || R <= 0 || S <= 0 || stride <= 0 || pad < 0)
                    return fail(HP_ERR_ARG, "layer %d: bad conv/FC geometry", i);
                int P = (inH + 2 * pad - R) / stride + 1;
                int Q = (inW + 2 * pad - S) / stride + 1;
                if (P <= 0 || Q <= 0) return fail(HP_ERR_ARG, "layer %d: empty output", i);
                nd.geo = ConvGeo{B, inH, inW, inC, L.K, R, S, P, Q, stride, pad};
                nd.H = P; nd.W = Q; nd.C = L.K;
                nd.w_off = off;
                nd.p_off = off;
                off += (size_t)L.K * R * S * inC;
                if (L.bias) { nd.b_off = off; off += L.K; }
                nd.p_cnt = off - nd.p_off;
                {
                    const int vw = st->dtype == HP_BF16 ? 8 : 4;
                    if (L.kind == HP_CONV && inC % vw != 0 && L.K % vw == 0) {
                        nd.padC = (inC + vw - 1) / vw * vw;
                        nd.geo_p = nd.geo;
                        nd.geo_p.C = nd.padC;
                    }
                }
                const ConvGeo& gfw = nd.padC ? nd.geo_p : nd.geo;
                nd.fwd = plan_gemm(OP_FWD, gfw, st->dtype, cus);
                nd.dgrad = plan_gemm(OP_DGRAD, nd.geo, st->dtype, cus);
                // fp32: the bias gradient rides along as a column of ones in the weight
                // gradient; bf16 would round dy there, so it is a separate fp32 sum
                nd.wgrad = plan_gemm(OP_WGRAD, gfw, st->dtype, cus,
                                     (L.bias && st->dtype == HP_FP32) ? 1 : 0);
                nd.bias_in_wgrad = nd.wgrad.bias_col != 0;
                // a small weight gradient (under 20 GFLOP) leaves most of the GPU
                // idle: it runs beside the data-gradient chain; a large one fills
                // the GPU by itself and stays in stream order
                // (not the fully connected kernel, which streams its output at the
                // rate of the whole device)
                nd.wgrad_side = 2.0 * nd.wgrad.M * nd.wgrad.Ncols * nd.wgrad.Kred < 2e10 &&
                                !nd.wgrad.fcw;
                size_t& wsw = nd.wgrad_side ? st->ws2_floats : st->ws_floats;
                if (L.bias && !nd.bias_in_wgrad)
                    wsw = std::max(wsw, colsum_ws_floats((long)B * P * Q, L.K));
                wsw = std::max(wsw, nd.wgrad.ws_floats);
                st->ws_floats = std::max({st->ws_floats, nd.fwd.ws_floats, nd.dgrad.ws_floats});
                break;
            }
            case HP_RELU:
                nd.H = nd.inH; nd.W = nd.inW; nd.C = nd.inC;
                break;
            case HP_MAXPOOL: {
                if (L.R <= 0 || L.S <= 0 || L.stride <= 0 || L.pad < 0 || L.pad >= L.R ||
                    L.pad >= L.S)
                    return fail(HP_ERR_ARG, "layer %d: bad pooling geometry", i);
                nd.H = (nd.inH + 2 * L.pad - L.R) / L.stride + 1;
                nd.W = (nd.inW + 2 * L.pad - L.S) / L.stride + 1;
                nd.C = nd.inC;
                if (nd.H <= 0 || nd.W <= 0) return fail(HP_ERR_ARG, "layer %d: empty output", i);
                break;
            }
            case HP_BN:
                if (L.C != nd.inC)
                    return fail(HP_ERR_ARG, "layer %d: BN expects %d channels, got %d", i, L.C, nd.inC);
                nd.H = nd.inH; nd.W = nd.inW; nd.C = nd.inC;
                nd.p_off = nd.w_off = off;
                off += L.C;
                nd.b_off = off;
                off += L.C;
                nd.p_cnt = 2 * (size_t)L.C;
                st->ws_floats = std::max(st->ws_floats, bn_ws_floats((long)B * nd.H * nd.W, L.C));
                break;
            case HP_ADD: {
                int h, w, c;
                if (L.in1 < -1 || L.in1 >= i || shape_of(st, L.in1, h, w, c) != HP_OK)
                    return fail(HP_ERR_ARG, "layer %d: bad second input %d", i, L.in1);
                if (h != nd.inH || w != nd.inW || c != nd.inC)
                    return fail(HP_ERR_ARG, "layer %d: residual add of mismatched shapes", i);
                if (L.in1 >= 0) st->nodes[L.in1].consumers++;
                nd.H = nd.inH; nd.W = nd.inW; nd.C = nd.inC;
                break;
            }
            case HP_GAP:
                nd.H = 1; nd.W = 1; nd.C = nd.inC;
                break;
            case HP_SOFTMAX_CE:
                if (i != n_layers - 1) return fail(HP_ERR_ARG, "loss head must be the last layer");
                if (L.in0 < 0) return fail(HP_ERR_ARG, "loss head needs logits from a layer");
                if (nd.inH * nd.inW * nd.inC != L.K)
                    return fail(HP_ERR_ARG, "layer %d: %d classes but %d logits", i, L.K,
                                nd.inH * nd.inW * nd.inC);
                nd.H = 1; nd.W = 1; nd.C = 0;
                st->has_loss = true;
                st->ws_floats = std::max(st->ws_floats, (size_t)B);
                break;
            default:
                return fail(HP_ERR_ARG, "layer %d: unknown kind %d", i, L.kind);
        }
        nd.out_elems = (size_t)B * nd.H * nd.W * nd.C;
    }
    st->P = off;
    // A residual add may hand its gradient buffer to an input that has other
    // consumers (the identity shortcut): that input's gradient then starts as
    // the add's gradient and its other consumers accumulate into the same
    // buffer.  Safe when the add's other input is a batch norm (its backward
    // only reads the buffer, on the stage stream) that every other consumer of
    // the shared input precedes: in reverse order the batch norm has read the
    // buffer before the first accumulation.
    for (int a = 0; a < n_layers; ++a) {
        Node& nd = st->nodes[a];
        if (nd.L.kind != HP_ADD) continue;
        for (int side = 0; side < 2; ++side) {
            const int j = side ? nd.L.in1 : nd.L.in0, k = side ? nd.L.in0 : nd.L.in1;
            if (j < 0 || k < 0 || j == k || st->nodes[j].consumers < 2 ||
                st->nodes[k].L.kind != HP_BN)
                continue;
            bool ok = true;
            for (int c = 0; c < n_layers && ok; ++c) {
                if (c == a) continue;
                const hp_layer& Lc = st->nodes[c].L;
                if (Lc.in0 == j || (Lc.kind == HP_ADD && Lc.in1 == j)) ok = c < k;
            }
            nd.add_share[side] = ok;
        }
    }
    // ReLU fusion: a ReLU reading a conv / FC / BN / add that has no other consumer
    for (int i = 0; i < n_layers; ++i) {
        Node& nd = st->nodes[i];
        if (nd.L.kind != HP_RELU || nd.L.in0 < 0) continue;
        Node& pr = st->nodes[nd.L.in0];
        int k = pr.L.kind;
        if ((k == HP_CONV || k == HP_FC || k == HP_BN || k == HP_ADD) && pr.consumers == 1 &&
            !pr.fuses_relu) {
            pr.fuses_relu = true;
            pr.relu_node = i;
            nd.relu_fused = true;
        }
    }
    // ReLU backward fused into the consumer's data-gradient write: a conv, FC or
    // max-pool reading a fused ReLU (producer conv / FC / add) that it alone reads
    for (int i = 0; i < n_layers; ++i) {
        Node& nd = st->nodes[i];
        int k = nd.L.kind;
        if ((k != HP_CONV && k != HP_FC && k != HP_MAXPOOL) || nd.L.in0 < 0) continue;
        Node& r = st->nodes[nd.L.in0];
        if (!r.relu_fused || r.consumers != 1) continue;
        if (st->nodes[r.L.in0].L.kind == HP_BN) continue;
        nd.mask_into = r.L.in0;
        r.bwd_by_consumer = true;
    }
    // device buffers
    st->node_bytes.assign(n_layers, 0);
    for (int i = 0; i < n_layers; ++i) {
        Node& nd = st->nodes[i];
        st->cur_node = i;
        if (nd.L.kind == HP_SOFTMAX_CE) continue;
        if (nd.relu_fused) {
            nd.y = st->nodes[nd.L.in0].y;
        } else {
            int rc = dev_alloc(st, &nd.y, nd.out_elems);
            if (rc) return rc;
        }
        int rc = dev_alloc(st, &nd.g, nd.out_elems);
        if (rc) return rc;
        if (nd.L.kind == HP_CONV && nd.consumers == 1) {
            int cons = -1;
            for (int c = i + 1; c < n_layers && cons < 0; ++c)
                if (st->nodes[c].L.in0 == i) cons = c;
            // a conv read only by a batch norm hands it its column statistics:
            // keep its forward on a kernel whose epilogue forms them
            if (cons >= 0 && st->nodes[cons].L.kind == HP_BN && nd.fwd.h16d) {
                nd.fwd = plan_gemm(OP_FWD, nd.padC ? nd.geo_p : nd.geo, st->dtype, num_cus(),
                                   0, 0);
                st->ws_floats = std::max(st->ws_floats, nd.fwd.ws_floats);
            }
            if (cons >= 0 && st->nodes[cons].L.kind == HP_BN &&
                plan_stats(nd.fwd, nd.L.bias ? EPI_BIAS : 0)) {
                nd.stats_rb = nd.fwd.bm;
                nd.stats_nb = (int)((nd.fwd.M + nd.fwd.bm - 1) / nd.fwd.bm);
                if ((rc = dev_alloc(st, &nd.stats, 2 * (size_t)nd.stats_nb * nd.C))) return rc;
            }
        }
        if (nd.padC) {
            const size_t xn = (size_t)st->batch * nd.inH * nd.inW * nd.padC;
            const size_t wn = (size_t)nd.L.K * nd.L.R * nd.L.S * nd.padC;
            if (st->dtype == HP_BF16) {
                if ((rc = dev_alloc16(st, &nd.xp16, xn)) || (rc = dev_alloc16(st, &nd.wp16, wn)))
                    return rc;
            } else if ((rc = dev_alloc(st, &nd.xp, xn)) || (rc = dev_alloc(st, &nd.wp, wn))) {
                return rc;
            }
            if ((rc = dev_alloc(st, &nd.dwp, wn))) return rc;
        }
        if (nd.L.kind == HP_MAXPOOL && nd.L.R * nd.L.S < 256 &&
            !maxpool_tiled(nd.inH, nd.inW, nd.L.R, nd.L.S, nd.L.stride, nd.L.pad, nd.H, nd.W)) {
            float* q = nullptr;
            if ((rc = dev_alloc(st, &q, (nd.out_elems + 3) / 4))) return rc;
            nd.arg = reinterpret_cast<uint8_t*>(q);
        }
        if (nd.L.kind == HP_BN) {
            if ((rc = dev_alloc(st, &nd.mean, nd.C))) return rc;
            if ((rc = dev_alloc(st, &nd.invstd, nd.C))) return rc;
        }
    }
    // bf16 operand copies for the contractions whose geometry allows them
    bool any16 = false;
    for (int i = 0; i < n_layers; ++i) {
        Node& nd = st->nodes[i];
        if ((nd.L.kind != HP_CONV && nd.L.kind != HP_FC) || !nd.fwd.h16) continue;
        any16 = true;
        const int j = nd.L.in0;
        st->cur_node = i;
        int rc = dev_alloc16(st, &nd.g16, nd.out_elems);
        st->cur_node = j;
        if (!rc && j < 0 && !st->x16)
            rc = dev_alloc16(st, &st->x16, (size_t)st->batch * st->H * st->W * st->C);
        else if (!rc && j >= 0 && !st->nodes[j].y16)
            rc = dev_alloc16(st, &st->nodes[j].y16, st->nodes[j].out_elems);
        if (rc) return rc;
    }
    st->cur_node = -1;
    if (any16) {
        int rc = dev_alloc16(st, &st->w16, st->P);
        if (rc) return rc;
        std::vector<WtLayer> tab;
        int tiles = 0;
        for (int i = 0; i < n_layers; ++i) {
            const Node& nd = st->nodes[i];
            if ((nd.L.kind != HP_CONV && nd.L.kind != HP_FC) || !nd.dgrad.h16k) continue;
            const ConvGeo& g = nd.geo;
            tab.push_back(WtLayer{(long)nd.w_off, g.K, g.R * g.S, g.C, tiles});
            tiles += wt_tiles(g.K, g.R * g.S, g.C);
        }
        if (!tab.empty()) {
            if ((rc = dev_alloc16(st, &st->w16t, st->P))) return rc;
            float* t = nullptr;
            const size_t tb = tab.size() * sizeof(WtLayer);
            if ((rc = dev_alloc(st, &t, (tb + 3) / 4))) return rc;
            HP_HIP(hipMemcpy(t, tab.data(), tb, hipMemcpyHostToDevice));
            st->wt_table = reinterpret_cast<WtLayer*>(t);
            st->wt_layers = (int)tab.size();
            st->wt_tiles_total = tiles;
        }
    }
    int rc = dev_alloc(st, &st->ws2, std::max<size_t>(st->ws2_floats, 64));
    if (rc) return rc;
    HP_HIP(hipStreamCreateWithFlags(&st->side, hipStreamNonBlocking));
    st->evs.resize(4, nullptr);
    for (auto& e : st->evs) HP_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    return dev_alloc(st, &st->ws, std::max<size_t>(st->ws_floats, 64));
}

int launch_ok(hipError_t e, const char* what, int layer) {
    if (e != hipSuccess)
        return fail(HP_ERR_HIP, "launch of %s (layer %d) failed: %s", what, layer,
                    hipGetErrorString(e));
    return HP_OK;
}

}  // namespace

// =================================================================== stage

extern "C" int hp_stage_create(const hp_layer* layers, int n_layers, int batch, int H, int W,
                               int C, int dtype_mode, void* stream, hp_stage** out) {
    if (!out) return fail(HP_ERR_ARG, "hp_stage_create: out is NULL");
    *out = nullptr;
    if (!layers || n_layers <= 0 || batch <= 0 || H <= 0 || W <= 0 || C <= 0)
        return fail(HP_ERR_ARG, "hp_stage_create: bad arguments");
    if (dtype_mode != HP_FP32 && dtype_mode != HP_BF16)
        return fail(HP_ERR_ARG, "hp_stage_create: unknown dtype mode %d", dtype_mode);
    hp_stage* st = new hp_stage();
    (void)hipGetDevice(&st->device);
    st->batch = batch; st->H = H; st->W = W; st->C = C;
    st->dtype = dtype_mode;
    st->stream = (hipStream_t)stream;
    int rc = build_stage(st, layers, n_layers);
    if (rc != HP_OK) {
        std::string msg = g_last_error;
        hp_stage_destroy(st);
        g_last_error = msg;
        return rc;
    }
    *out = st;
    return HP_OK;
}

extern "C" int hp_stage_destroy(hp_stage* st) {
    if (!st) return HP_OK;
    if (st->stream || !st->allocs.empty()) (void)hipStreamSynchronize(st->stream);
    if (st->side) (void)hipStreamSynchronize(st->side);
    for (auto e : st->evs)
        if (e) (void)hipEventDestroy(e);
    if (st->side) (void)hipStreamDestroy(st->side);
    for (void* p : st->allocs) (void)hipFree(p);
    delete st;
    return HP_OK;
}

extern "C" int hp_stage_param_count(const hp_stage* st, size_t* count) {
    if (!st || !count) return fail(HP_ERR_ARG, "hp_stage_param_count: NULL argument");
    *count = st->P;
    return HP_OK;
}

extern "C" int hp_stage_param_layout(const hp_stage* st, int layer, size_t* offset, size_t* count) {
    if (!st || !offset || !count) return fail(HP_ERR_ARG, "hp_stage_param_layout: NULL argument");
    if (layer < 0 || layer >= (int)st->nodes.size())
        return fail(HP_ERR_ARG, "hp_stage_param_layout: no layer %d", layer);
    *offset = st->nodes[layer].p_cnt ? st->nodes[layer].p_off : 0;
    *count = st->nodes[layer].p_cnt;
    return HP_OK;
}

extern "C" int hp_stage_output_shape(const hp_stage* st, int layer, int dims[3]) {
    if (!st || !dims) return fail(HP_ERR_ARG, "hp_stage_output_shape: NULL argument");
    int n = (int)st->nodes.size();
    if (layer == -1) layer = st->has_loss ? n - 2 : n - 1;
    if (layer < 0 || layer >= n) return fail(HP_ERR_ARG, "hp_stage_output_shape: no layer %d", layer);
    const Node& nd = st->nodes[layer];
    dims[0] = nd.H; dims[1] = nd.W; dims[2] = nd.C;
    return HP_OK;
}

extern "C" int hp_stage_device_bytes(const hp_stage* st, size_t* bytes) {
    if (!st || !bytes) return fail(HP_ERR_ARG, "hp_stage_device_bytes: NULL argument");
    *bytes = st->bytes;
    return HP_OK;
}

extern "C" int hp_stage_set_timing(hp_stage* st, int enable) {
    if (!st) return fail(HP_ERR_ARG, "hp_stage_set_timing: NULL stage");
    st->timer.on = enable != 0;
    return HP_OK;
}

namespace {

// Sums the recorded event pairs per category (after synchronising `s`) and
// returns the events to the pool.
int read_timer(StageTimer& tm, hipStream_t s, int ncat, double* ms, int64_t* launches) {
    HP_HIP(hipStreamSynchronize(s));
    for (int i = 0; i < ncat; ++i) { ms[i] = 0.0; launches[i] = 0; }
    for (auto& r : tm.recs) {
        float t = 0.f;
        HP_HIP(hipEventElapsedTime(&t, r.a, r.b));
        if (r.cat >= 0 && r.cat < ncat) { ms[r.cat] += t; launches[r.cat] += 1; }
        tm.pool.push_back(r.a);
        tm.pool.push_back(r.b);
    }
    tm.recs.clear();
    return HP_OK;
}

}  // namespace

extern "C" int hp_stage_read_timing(hp_stage* st, double ms[2], int64_t launches[2]) {
    if (!st || !ms || !launches) return fail(HP_ERR_ARG, "hp_stage_read_timing: NULL argument");
    return read_timer(st->timer, st->stream, 2, ms, launches);
}

extern "C" int hp_stage_layer_bytes(const hp_stage* st, size_t* bytes, int n) {
    if (!st || !bytes) return fail(HP_ERR_ARG, "hp_stage_layer_bytes: NULL argument");
    const int nl = (int)st->nodes.size();
    if (n != nl + 1)
        return fail(HP_ERR_ARG, "hp_stage_layer_bytes: n = %d, the stage needs %d", n, nl + 1);
    for (int i = 0; i < nl; ++i) bytes[i] = st->node_bytes[i];
    bytes[nl] = st->shared_bytes;
    return HP_OK;
}

extern "C" int hp_stage_read_layer_timing(hp_stage* st, double* fwd_ms, double* bwd_ms, int n) {
    if (!st || !fwd_ms || !bwd_ms) return fail(HP_ERR_ARG, "hp_stage_read_layer_timing: NULL argument");
    const int nl = (int)st->nodes.size();
    if (n != nl + 1)
        return fail(HP_ERR_ARG, "hp_stage_read_layer_timing: n = %d, the stage needs %d", n, nl + 1);
    HP_HIP(hipStreamSynchronize(st->stream));
    for (int i = 0; i < n; ++i) fwd_ms[i] = bwd_ms[i] = 0.0;
    StageTimer& tm = st->timer;
    for (auto& r : tm.recs) {
        float t = 0.f;
        HP_HIP(hipEventElapsedTime(&t, r.a, r.b));
        const int slot = (r.node >= 0 && r.node < nl) ? r.node : nl;
        (r.phase ? bwd_ms : fwd_ms)[slot] += t;
        tm.pool.push_back(r.a);
        tm.pool.push_back(r.b);
    }
    tm.recs.clear();
    return HP_OK;
}

extern "C" int hp_stage_forward(hp_stage* st, const float* w, const float* x, float* y,
                                const int32_t* labels, float* loss) {
    if (!st || !x || (!w && st->P)) return fail(HP_ERR_ARG, "hp_stage_forward: NULL argument");
    if (st->has_loss && (!labels || !loss))
        return fail(HP_ERR_ARG, "hp_stage_forward: loss head needs labels and loss");
    if (!st->has_loss && (labels || loss))
        return fail(HP_ERR_ARG, "hp_stage_forward: stage has no loss head");
    if (!st->has_loss && !y) return fail(HP_ERR_ARG, "hp_stage_forward: y is NULL");
    hipStream_t s = st->stream;
    const int B = st->batch;
    st->x16_ready = false;
    for (Node& nd : st->nodes) nd.y16_ready = false;
    st->timer.node = -1;
    st->timer.phase = 0;
    if (st->w16) {
        st->timer.begin(1, s);
        hipError_t e = launch_cast_bf16(w, st->w16, st->P, s);
        if (e == hipSuccess && st->w16t)
            e = launch_cast_bf16_t(w, st->w16t, st->wt_table, st->wt_layers,
                                   st->wt_tiles_total, s);
        st->timer.end(s);
        int rc = launch_ok(e, "weight cast", -1);
        if (rc) return rc;
    }
    for (size_t i = 0; i < st->nodes.size(); ++i) {
        Node& nd = st->nodes[i];
        const hp_layer& L = nd.L;
        const float* in = L.in0 < 0 ? x : st->nodes[L.in0].y;
        st->timer.node = (int)i;
        hipError_t e = hipSuccess;
        StageTimer& tm = st->timer;
        const uint16_t* in16 = nullptr;
        if ((L.kind == HP_CONV || L.kind == HP_FC) && nd.fwd.h16 && st->w16 && !nd.padC) {
            // bf16 copy of the input value, made by its first contraction consumer
            in16 = L.in0 < 0 ? st->x16 : st->nodes[L.in0].y16;
            bool& ready = L.in0 < 0 ? st->x16_ready : st->nodes[L.in0].y16_ready;
            if (!ready) {
                const size_t n_in = L.in0 < 0 ? (size_t)B * st->H * st->W * st->C
                                              : st->nodes[L.in0].out_elems;
                tm.begin(1, s);
                e = launch_cast_bf16(in, const_cast<uint16_t*>(in16), n_in, s);
                tm.end(s);
                int rc = launch_ok(e, "activation cast", (int)i);
                if (rc) return rc;
                ready = true;
            }
        }
        // producers that can write the bf16 copy of the value they make (the
        // ReLU node's value when they apply their consumer ReLU)
        uint16_t* out16 = nullptr;
        if (L.kind == HP_BN || L.kind == HP_ADD || L.kind == HP_MAXPOOL) {
            Node& vis = nd.fuses_relu ? st->nodes[nd.relu_node] : nd;
            if (vis.y16) {
                out16 = vis.y16;
                vis.y16_ready = true;
            }
        }
        // a ReLU applied in its producer's epilogue launches nothing: no record
        const bool launches = !(L.kind == HP_RELU && nd.relu_fused);
        if (launches) tm.begin(L.kind == HP_CONV || L.kind == HP_FC ? 0 : 1, s);
        switch (L.kind) {
            case HP_CONV:
            case HP_FC: {
                Epilogue ep;
                ep.flags = (L.bias ? EPI_BIAS : 0) | (nd.fuses_relu ? EPI_RELU : 0);
                ep.bias = L.bias ? w + nd.b_off : nullptr;
                ep.stats = nd.stats;
                // the bf16 copy a consuming contraction reads (of the ReLU's
                // value when this layer applies it) comes from the epilogue
                Node& vis = nd.fuses_relu ? st->nodes[nd.relu_node] : nd;
                if (vis.y16 && !nd.stats) {
                    ep.out16 = vis.y16;
                    vis.y16_ready = true;
                }
                if (nd.padC) {
                    // zero-padded copies of the input and the weights, then the
                    // contraction on the padded geometry
                    const int C0 = nd.geo.C, Cp = nd.padC;
                    const size_t xr = (size_t)B * nd.inH * nd.inW;
                    const size_t wr = (size_t)L.K * L.R * L.S;
                    e = launch_pad_channels(in, nd.xp, nd.xp16, xr, C0, Cp, s);
                    if (e == hipSuccess)
                        e = launch_pad_channels(w + nd.w_off, nd.wp, nd.wp16, wr, C0, Cp, s);
                    if (e == hipSuccess)
                        e = launch_gemm(nd.fwd, nd.geo_p, nd.xp ? nd.xp : in, nd.wp ? nd.wp : w,
                                        nd.y, ep, st->ws, s, nd.xp16, nd.wp16);
                    break;
                }
                e = launch_gemm(nd.fwd, nd.geo, in, w + nd.w_off, nd.y, ep, st->ws, s, in16,
                                in16 ? st->w16 + nd.w_off : nullptr);
                break;
            }
            case HP_RELU:
                if (!nd.relu_fused) e = launch_relu_fwd(in, nd.y, nd.out_elems, s);
                break;
            case HP_MAXPOOL:
                e = launch_maxpool_fwd(in, nd.y, B, nd.inH, nd.inW, nd.inC, L.R, L.S, L.stride,
                                       L.pad, nd.H, nd.W, s, out16, nd.arg);
                break;
            case HP_BN: {
                const Node* pc = L.in0 >= 0 ? &st->nodes[L.in0] : nullptr;
                if (pc && pc->stats)       // statistics from the producing contraction
                    e = launch_bn_fwd_partials(in, (long)B * nd.H * nd.W, nd.C, w + nd.w_off,
                                               w + nd.b_off, L.eps, nd.y, nd.mean, nd.invstd,
                                               nd.fuses_relu ? 1 : 0, pc->stats,
                                               pc->stats + (size_t)pc->stats_nb * nd.C,
                                               pc->stats_nb, pc->stats_rb, s, out16);
                else
                    e = launch_bn_fwd(in, (long)B * nd.H * nd.W, nd.C, w + nd.w_off, w + nd.b_off,
                                      L.eps, nd.y, nd.mean, nd.invstd, nd.fuses_relu ? 1 : 0,
                                      st->ws, s, out16);
                break;
            }
            case HP_ADD: {
                const float* in1 = L.in1 < 0 ? x : st->nodes[L.in1].y;
                e = launch_add_fwd(in, in1, nd.y, nd.out_elems, nd.fuses_relu ? 1 : 0, s, out16);
                break;
            }
            case HP_GAP:
                e = launch_gap_fwd(in, nd.y, B, nd.inH * nd.inW, nd.C, s);
                break;
            case HP_SOFTMAX_CE: {
                // dz goes straight into the logits' gradient buffer
                Node& lg = st->nodes[L.in0];
                e = launch_softmax_ce(in, labels, B, L.K, loss, lg.g, st->ws, s);
                if (e == hipSuccess && y)
                    e = hipMemcpyAsync(y, in, (size_t)B * L.K * sizeof(float),
                                       hipMemcpyDeviceToDevice, s);
                break;
            }
        }
        if (launches) tm.end(s);
        int rc = launch_ok(e, "forward", (int)i);
        if (rc) return rc;
    }
    if (!st->has_loss) {
        Node& last = st->nodes.back();
        HP_HIP(hipMemcpyAsync(y, last.y, last.out_elems * sizeof(float), hipMemcpyDeviceToDevice, s));
    }
    st->fwd_w = w;
    st->fwd_x = x;
    st->fwd_done = true;
    return HP_OK;
}

namespace {

// The backward pass with the workspaces of the stage stream (ws) and of the
// weight-gradient stream (ws2) given by the caller: the stage's own, or the
// library's static scratch (hp_stage_backward_noalloc).
int stage_backward(hp_stage* st, const float* w, const float* dy, float* dx, float* grad,
                   float* ws, float* ws2) {
    if (!st || !grad || (!w && st->P)) return fail(HP_ERR_ARG, "hp_stage_backward: NULL argument");
    if (!st->fwd_done) return fail(HP_ERR_STATE, "hp_stage_backward: no forward pass to differentiate");
    if (w != st->fwd_w)
        return fail(HP_ERR_STATE, "hp_stage_backward: weights differ from the forward pass");
    if (st->has_loss && dy) return fail(HP_ERR_ARG, "hp_stage_backward: loss stage takes no dy");
    if (!st->has_loss && !dy) return fail(HP_ERR_ARG, "hp_stage_backward: dy is NULL");
    hipStream_t s = st->stream;
    const int B = st->batch;
    const int n = (int)st->nodes.size();
    const float* x = st->fwd_x;
    for (Node& nd : st->nodes) {
        nd.g_written = false;
        nd.g_alias = nullptr;
        nd.g_shared = false;
        nd.g_final = nullptr;
    }
    st->bwd_dx = nullptr;
    bool dx_written = false;
    for (Node& nd : st->nodes) nd.g16_ready = false;
    // `a` happens before everything enqueued on `b` afterwards
    auto order = [&](hipStream_t a, hipStream_t b) -> hipError_t {
        hipEvent_t e = st->evs[st->ev_next++ % st->evs.size()];
        hipError_t r = hipEventRecord(e, a);
        return r == hipSuccess ? hipStreamWaitEvent(b, e, 0) : r;
    };
    if (st->has_loss) st->nodes[st->nodes.back().L.in0].g_written = true;  // dz from forward

    // destination of a gradient sent to value j: (pointer, accumulate?)
    auto dest = [&](int j, float** p, int* acc) -> bool {
        if (j < 0) {
            if (!dx) return false;
            *p = dx;
            *acc = dx_written ? 1 : 0;
            dx_written = true;
            return true;
        }
        if (st->nodes[j].g_shared) {           // accumulate into the shared buffer
            *p = const_cast<float*>(st->nodes[j].g_alias);
            *acc = 1;
            return true;
        }
        *p = st->nodes[j].g;
        *acc = st->nodes[j].g_written ? 1 : 0;
        st->nodes[j].g_written = true;
        return true;
    };

    // the bf16 copy of value j's gradient, which j's own contractions read,
    // written by the layer that sends j its gradient when that is the only
    // contribution (j has one consumer and nothing was written before)
    auto sole_grad16 = [&](int j, int acc) -> uint16_t* {
        if (j < 0 || acc) return nullptr;
        Node& t = st->nodes[j];
        if (!t.g16 || t.consumers != 1 || t.g_shared) return nullptr;
        t.g16_ready = true;
        return t.g16;
    };

    st->timer.phase = 1;
    for (int i = n - 1; i >= 0; --i) {
        Node& nd = st->nodes[i];
        const hp_layer& L = nd.L;
        st->timer.node = i;
        if (L.kind == HP_SOFTMAX_CE) continue;
        const float* gin;
        if (i == n - 1 && !st->has_loss) gin = dy;
        else if (nd.g_alias) gin = nd.g_alias;
        else if (nd.g_written) gin = nd.g;
        else continue;   // no gradient reaches this value
        // complete now (every consumer is done); a batch norm that applies its
        // consumer ReLU receives the ReLU's unmasked gradient instead
        nd.g_final = (L.kind == HP_BN && nd.fuses_relu) ? nullptr : gin;
        const float* in = L.in0 < 0 ? x : st->nodes[L.in0].y;
        hipError_t e = hipSuccess;
        float* d;
        int acc;
        const bool gemm_node = L.kind == HP_CONV || L.kind == HP_FC;
        if (!gemm_node) st->timer.begin(1, s);
        switch (L.kind) {
            case HP_CONV:
            case HP_FC: {
                StageTimer& tm = st->timer;
                const uint16_t* in16 = nullptr;
                const uint16_t* g16 = nullptr;
                if (nd.fwd.h16 && st->w16) {
                    in16 = nd.padC ? nd.xp16 : L.in0 < 0 ? st->x16 : st->nodes[L.in0].y16;
                    if (!nd.g16_ready) {
                        tm.begin(1, s);
                        e = launch_cast_bf16(gin, nd.g16, nd.out_elems, s);
                        tm.end(s);
                    }
                    g16 = nd.g16;
                }
                // weight gradient (and a separate bias column sum), on the side
                // stream once gin and its bf16 copy are complete
                hipStream_t sd = nd.wgrad_side ? st->side : s;
                float* wsw = nd.wgrad_side ? ws2 : ws;
                if (e == hipSuccess && nd.wgrad_side) e = order(s, sd);
                tm.begin(0, sd);
                Epilogue wep;                     // bias gradient = appended column
                wep.bias_out = nd.bias_in_wgrad ? grad + nd.b_off : nullptr;
                if (e == hipSuccess && nd.padC) {
                    // on the padded geometry, then compacted into grad
                    e = launch_gemm(nd.wgrad, nd.geo_p, nd.xp ? nd.xp : in, gin, nd.dwp, wep, wsw,
                                    sd, in16, g16);
                    if (e == hipSuccess)
                        e = launch_unpad_channels(nd.dwp, grad + nd.w_off,
                                                  (size_t)L.K * L.R * L.S, nd.geo.C, nd.padC, sd);
                } else if (e == hipSuccess) {
                    e = launch_gemm(nd.wgrad, nd.geo, in, gin, grad + nd.w_off, wep, wsw, sd,
                                    in16, g16);
                }
                tm.end(sd);
                if (e == hipSuccess && L.bias && !nd.bias_in_wgrad) {
                    tm.begin(1, sd);
                    e = launch_colsum(gin, (long)B * nd.H * nd.W, nd.C, grad + nd.b_off, wsw, sd);
                    tm.end(sd);
                }
                const int tgt = nd.mask_into >= 0 ? nd.mask_into : L.in0;
                if (e == hipSuccess && dest(tgt, &d, &acc)) {
                    Epilogue dep;
                    dep.flags = acc ? EPI_ACCUM : 0;
                    if (nd.mask_into >= 0) {
                        dep.flags |= EPI_MASK;
                        dep.mask = st->nodes[L.in0].y;
                    }
                    dep.out16 = sole_grad16(tgt, acc);
                    tm.begin(0, s);
                    e = launch_gemm(nd.dgrad, nd.geo, gin, w + nd.w_off, d, dep, ws, s, g16,
                                    g16 ? st->w16 + nd.w_off : nullptr,
                                    g16 && st->w16t ? st->w16t + nd.w_off : nullptr);
                    tm.end(s);
                }
                break;
            }
            case HP_RELU: {
                const bool into_bn = nd.relu_fused && st->nodes[L.in0].L.kind == HP_BN;
                if (nd.bwd_by_consumer) {
                    // already applied by the consumer's data-gradient write
                    st->timer.cancel();
                } else if (into_bn) {
                    // the BN backward applies the ReLU mask itself: hand it this gradient
                    Node& pr = st->nodes[L.in0];
                    pr.g_alias = gin;
                    pr.g_written = true;
                    st->timer.cancel();
                } else if (dest(L.in0, &d, &acc)) {
                    e = launch_relu_bwd(nd.y, gin, d, nd.out_elems, acc, s);
                }
                break;
            }
            case HP_MAXPOOL: {
                const int tgt = nd.mask_into >= 0 ? nd.mask_into : L.in0;
                const float* mask = nd.mask_into >= 0 ? st->nodes[L.in0].y : nullptr;
                if (dest(tgt, &d, &acc))
                    e = launch_maxpool_bwd(in, gin, d, B, nd.inH, nd.inW, nd.inC, L.R, L.S,
                                           L.stride, L.pad, nd.H, nd.W, acc, mask, s, nd.arg,
                                           sole_grad16(tgt, acc));
                break;
            }
            case HP_BN: {
                // with a fused ReLU, nd.y holds the ReLU output and serves as the mask
                bool want = dest(L.in0, &d, &acc);
                // the producing conv reads this gradient as a bf16 operand: write
                // that copy too when this BN is the conv's only consumer
                uint16_t* d16 = nullptr;
                if (want && L.in0 >= 0 && st->w16) {
                    Node& pc = st->nodes[L.in0];
                    if ((pc.L.kind == HP_CONV || pc.L.kind == HP_FC) && pc.fwd.h16 &&
                        pc.consumers == 1) {
                        d16 = pc.g16;
                        pc.g16_ready = true;
                    }
                }
                e = launch_bn_bwd(in, gin, nd.fuses_relu ? nd.y : nullptr, (long)B * nd.H * nd.W,
                                  nd.C, w + nd.w_off, nd.mean, nd.invstd, want ? d : nullptr,
                                  grad + nd.w_off, grad + nd.b_off, want ? acc : 0, ws, s, d16);
                break;
            }
            case HP_ADD: {
                // both inputs receive this gradient unchanged.  An input that
                // nothing else reads takes it as its own without a copy (its
                // backward only reads it; the layers that wrote it are done),
                // unless it is the caller's dy.
                bool copied = false;
                auto route = [&](int j, int side) -> hipError_t {
                    if (j >= 0 && gin != dy && st->nodes[j].consumers == 1 &&
                        !st->nodes[j].g_written) {
                        st->nodes[j].g_alias = gin;
                        st->nodes[j].g_written = true;
                        return hipSuccess;
                    }
                    if (j >= 0 && nd.add_share[side] && gin == nd.g && !st->nodes[j].g_written) {
                        st->nodes[j].g_alias = gin;       // the identity shortcut's gradient
                        st->nodes[j].g_written = true;
                        st->nodes[j].g_shared = true;
                        nd.g_final = nullptr;             // the buffer now accumulates j's
                        return hipSuccess;
                    }
                    if (dest(j, &d, &acc)) {
                        copied = true;
                        return launch_copy_or_acc(gin, d, nd.out_elems, acc, s);
                    }
                    return hipSuccess;
                };
                e = route(L.in0, 0);
                if (e == hipSuccess) e = route(L.in1, 1);
                if (!copied) st->timer.cancel();    // both inputs took the buffer
                break;
            }
            case HP_GAP:
                if (dest(L.in0, &d, &acc))
                    e = launch_gap_bwd(gin, d, B, nd.inH * nd.inW, nd.C, acc, s);
                break;
        }
        if (!gemm_node) st->timer.end(s);
        int rc = launch_ok(e, "backward", i);
        if (rc) return rc;
    }
    // a buffer handed to an identity shortcut as its shared gradient went on
    // accumulating the shortcut's other consumers after the layers that only
    // read it (the add, the add's other input) were done with it
    for (const Node& a : st->nodes)
        if (a.g_shared && a.g_alias)
            for (Node& b : st->nodes)
                if (&b != &a && b.g_final == a.g_alias) b.g_final = nullptr;
    // the caller's stream sees the complete gradient
    HP_HIP(order(st->side, s));
    st->fwd_done = false;
    st->bwd_dx = dx_written ? dx : nullptr;
    return HP_OK;
}

}  // namespace

extern "C" int hp_stage_backward(hp_stage* st, const float* w, const float* dy, float* dx,
                                 float* grad) {
    if (!st) return fail(HP_ERR_ARG, "hp_stage_backward: NULL stage");
    return stage_backward(st, w, dy, dx, grad, st->ws, st->ws2);
}

// ------------------------------------------- backward pass without allocation
//
// The workspaces of hp_stage_backward_noalloc: one static array per device
// (each GPU the library runs on holds its own copy until the process ends).
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is taken once per device with hipGetSymbolAddress, with that
// device current, and only that address is ever handed to kernels.
constexpr size_t HP_SCRATCH_BYTES = HP_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[HP_SCRATCH_BYTES];

namespace {

constexpr int HP_MAX_DEVICES = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[HP_MAX_DEVICES] = {};

// Device address of `scratch` on the current device (set up on first use).
int scratch_address(int dev, void** out) {
    if (dev < 0 || dev >= HP_MAX_DEVICES)
        return fail(HP_ERR_ARG, "hp_stage_backward_noalloc: device %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(HP_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return HP_OK;
}

}  // namespace

extern "C" int hp_stage_backward_noalloc(hp_stage* st, const float* w, const float* dy,
                                         float* dx, float* grad) {
    if (!st) return fail(HP_ERR_ARG, "hp_stage_backward_noalloc: NULL stage");
    // the stage's stream workspace, then the weight-gradient stream's, each
    // starting on a 256-byte boundary
    const size_t ws_bytes = round_up(std::max<size_t>(st->ws_floats, 64) * sizeof(float), 256);
    const size_t ws2_bytes = round_up(std::max<size_t>(st->ws2_floats, 64) * sizeof(float), 256);
    if (ws_bytes + ws2_bytes > HP_SCRATCH_BYTES)
        return fail(HP_ERR_ARG,
                    "hp_stage_backward_noalloc: the stage needs %zu bytes of workspace, the "
                    "static scratch holds %zu",
                    ws_bytes + ws2_bytes, HP_SCRATCH_BYTES);
    int cur = -1;
    HP_HIP(hipGetDevice(&cur));
    if (cur != st->device)
        return fail(HP_ERR_STATE,
                    "hp_stage_backward_noalloc: device %d is current, the stage lives on %d",
                    cur, st->device);
    void* base = nullptr;
    int rc = scratch_address(cur, &base);
    if (rc) return rc;
    float* ws = static_cast<float*>(base);
    float* ws2 = reinterpret_cast<float*>(static_cast<unsigned char*>(base) + ws_bytes);
    return stage_backward(st, w, dy, dx, grad, ws, ws2);
}

extern "C" int hp_stage_layer_buffers(const hp_stage* st, int layer, const float** value,
                                      const float** grad) {
    if (!st || !value || !grad) return fail(HP_ERR_ARG, "hp_stage_layer_buffers: NULL argument");
    const int n = (int)st->nodes.size();
    if (layer < -1 || layer >= n)
        return fail(HP_ERR_ARG, "hp_stage_layer_buffers: no layer %d", layer);
    if (layer == -1) {
        *value = st->fwd_x;
        *grad = st->bwd_dx;
        return HP_OK;
    }
    const Node& nd = st->nodes[layer];
    *value = (nd.L.kind == HP_SOFTMAX_CE || nd.fuses_relu) ? nullptr : nd.y;
    *grad = nd.g_final;
    return HP_OK;
}

// ======================================================== parameter server

extern "C" int hp_ps_create(size_t P, const float* w0, int N, int D, void* stream, hp_ps** out) {
    if (!out) return fail(HP_ERR_ARG, "hp_ps_create: out is NULL");
    *out = nullptr;
    if (P == 0 || !w0 || N <= 0 || D < 0) return fail(HP_ERR_ARG, "hp_ps_create: bad arguments");
    hp_ps* ps = new hp_ps();
    ps->P = P; ps->N = N; ps->D = D;
    ps->stream = (hipStream_t)stream;
    ps->clock.assign(N, 0);
    ps->pushed.assign(N, 0);
    ps->vws.assign(N, nullptr);
    hipError_t e = hipMalloc(&ps->wg, round_up(P, 64) * sizeof(float));
    if (e != hipSuccess) {
        delete ps;
        return fail(e == hipErrorOutOfMemory ? HP_ERR_NOMEM : HP_ERR_HIP, "hp_ps_create: %s",
                    hipGetErrorString(e));
    }
    e = launch_wsp_copy(w0, ps->wg, P, ps->stream);
    if (e != hipSuccess) {
        (void)hipFree(ps->wg);
        delete ps;
        return fail(HP_ERR_HIP, "hp_ps_create: copy failed: %s", hipGetErrorString(e));
    }
    *out = ps;
    return HP_OK;
}

extern "C" int hp_ps_destroy(hp_ps* ps) {
    if (!ps) return HP_OK;
    for (hp_vw* v : ps->vws)
        if (v) v->ps = nullptr;
    (void)hipStreamSynchronize(ps->stream);
    (void)hipFree(ps->wg);
    delete ps;
    return HP_OK;
}

extern "C" int hp_ps_weights(const hp_ps* ps, const float** wg) {
    if (!ps || !wg) return fail(HP_ERR_ARG, "hp_ps_weights: NULL argument");
    *wg = ps->wg;
    return HP_OK;
}

extern "C" int hp_ps_clock(const hp_ps* ps, int* c_global) {
    if (!ps || !c_global) return fail(HP_ERR_ARG, "hp_ps_clock: NULL argument");
    *c_global = ps->cg;
    return HP_OK;
}

extern "C" int hp_ps_set_timing(hp_ps* ps, int enable) {
    if (!ps) return fail(HP_ERR_ARG, "hp_ps_set_timing: NULL server");
    ps->timer.on = enable != 0;
    return HP_OK;
}

extern "C" int hp_ps_read_timing(hp_ps* ps, double ms[6], int64_t launches[6]) {
    if (!ps || !ms || !launches) return fail(HP_ERR_ARG, "hp_ps_read_timing: NULL argument");
    return read_timer(ps->timer, ps->stream, 6, ms, launches);
}

// ========================================================== virtual worker

extern "C" int hp_vw_create(hp_ps* ps, int id, int s_local, hp_vw** out) {
    if (!out) return fail(HP_ERR_ARG, "hp_vw_create: out is NULL");
    *out = nullptr;
    if (!ps || id < 0 || id >= ps->N || s_local < 0)
        return fail(HP_ERR_ARG, "hp_vw_create: bad arguments");
    if (ps->vws[id]) return fail(HP_ERR_STATE, "hp_vw_create: VW %d already exists", id);
    hp_vw* v = new hp_vw();
    v->ps = ps;
    v->id = id;
    v->W = s_local + 1;
    v->P = ps->P;
    v->stride = round_up(ps->P, 64);     // 256-byte aligned ring slots
    hipError_t e = hipMalloc(&v->ring, (size_t)v->W * v->stride * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(&v->ut, v->stride * sizeof(float));
    if (e != hipSuccess) {
        if (v->ring) (void)hipFree(v->ring);
        delete v;
        return fail(e == hipErrorOutOfMemory ? HP_ERR_NOMEM : HP_ERR_HIP, "hp_vw_create: %s",
                    hipGetErrorString(e));
    }
    // w_1 = ... = w_W = the server's current weights
    for (int s = 0; s < v->W && e == hipSuccess; ++s)
        e = launch_wsp_copy(ps->wg, v->ring + (size_t)s * v->stride, v->P, ps->stream);
    if (e != hipSuccess) {
        (void)hipFree(v->ring);
        (void)hipFree(v->ut);
        delete v;
        return fail(HP_ERR_HIP, "hp_vw_create: copy failed: %s", hipGetErrorString(e));
    }
    v->V.assign(v->W, std::vector<int64_t>(ps->N, 0));
    for (int n = 0; n < ps->N; ++n) {
        // a VW created after others pushed starts from w_g and its contents
        for (int s = 0; s < v->W; ++s) v->V[s][n] = (int64_t)v->W * ps->pushed[n];
    }
    ps->vws[id] = v;
    *out = v;
    return HP_OK;
}

extern "C" int hp_vw_destroy(hp_vw* v) {
    if (!v) return HP_OK;
    if (v->ps) {
        (void)hipStreamSynchronize(v->ps->stream);
        v->ps->vws[v->id] = nullptr;
    } else {
        (void)hipDeviceSynchronize();
    }
    (void)hipFree(v->ring);
    (void)hipFree(v->ut);
    if (v->vel) (void)hipFree(v->vel);
    delete v;
    return HP_OK;
}

extern "C" int hp_vw_set_momentum(hp_vw* v, float mu) {
    if (!v) return fail(HP_ERR_ARG, "hp_vw_set_momentum: NULL VW");
    if (!v->ps) return fail(HP_ERR_STATE, "hp_vw_set_momentum: parameter server destroyed");
    if (!(mu >= 0.f && mu < 1.f))
        return fail(HP_ERR_ARG, "hp_vw_set_momentum: momentum %g outside [0, 1)", (double)mu);
    if (v->inflight)
        return fail(HP_ERR_STATE, "hp_vw_set_momentum: VW %d has minibatches in flight", v->id);
    if (mu != 0.f && !v->vel) {
        hipError_t e = hipMalloc(&v->vel, v->stride * sizeof(float));
        if (e != hipSuccess)
            return fail(e == hipErrorOutOfMemory ? HP_ERR_NOMEM : HP_ERR_HIP,
                        "hp_vw_set_momentum: %s", hipGetErrorString(e));
    }
    if (v->vel) HP_HIP(hipMemsetAsync(v->vel, 0, v->stride * sizeof(float), v->ps->stream));
    v->mu = mu;
    return HP_OK;
}

extern "C" int hp_wsp_weights(hp_vw* v, const float** w) {
    if (!v || !w) return fail(HP_ERR_ARG, "hp_wsp_weights: NULL argument");
    if (!v->ps) return fail(HP_ERR_STATE, "hp_wsp_weights: parameter server destroyed");
    if (v->push_due) return fail(HP_ERR_STATE, "hp_wsp_weights: wave %d not pushed yet", v->c);
    if (v->need_pull)
        return fail(HP_ERR_STATE, "hp_wsp_weights: VW %d is gated by the clock bound", v->id);
    if (v->inflight >= v->W)
        return fail(HP_ERR_STATE, "hp_wsp_weights: VW %d already has %d minibatches in flight",
                    v->id, v->inflight);
    int slot = (int)((v->p + v->inflight) % v->W);
    *w = v->ring + (size_t)slot * v->stride;
    v->inflight += 1;
    return HP_OK;
}

extern "C" int hp_wsp_local_update(hp_vw* v, const float* grad, float lr) {
    if (!v || !grad) return fail(HP_ERR_ARG, "hp_wsp_local_update: NULL argument");
    if (!v->ps) return fail(HP_ERR_STATE, "hp_wsp_local_update: parameter server destroyed");
    if (v->inflight == 0)
        return fail(HP_ERR_STATE, "hp_wsp_local_update: no minibatch was started (hp_wsp_weights)");
    // a completed wave is pushed, and its gate passed, before the next
    // minibatch completes: the first update of a wave overwrites u~, and the
    // pull writes the ring slot the next completion would write
    if (v->push_due)
        return fail(HP_ERR_STATE, "hp_wsp_local_update: wave %d of VW %d not pushed yet",
                    (int)(v->p / v->W) - 1, v->id);
    if (v->need_pull)
        return fail(HP_ERR_STATE, "hp_wsp_local_update: VW %d is gated by the clock bound", v->id);
    const int64_t q = v->p + 1;
    const int W = v->W;
    const int slot = (int)((q - 1) % W);
    const int newest = (int)((q - 2 + W) % W);
    const int first = ((q - 1) % W) == 0;
    StageTimer& tm = v->ps->timer;
    tm.begin(first ? 0 : 1, v->ps->stream);
    hipError_t e = v->mu != 0.f
        ? launch_wsp_local_update_momentum(grad, v->ring + (size_t)newest * v->stride,
                                           v->ring + (size_t)slot * v->stride, v->ut, v->vel,
                                           v->P, lr, v->mu, first, v->ps->stream)
        : launch_wsp_local_update(grad, v->ring + (size_t)newest * v->stride,
                                  v->ring + (size_t)slot * v->stride, v->ut, v->P, lr, first,
                                  v->ps->stream);
    tm.end(v->ps->stream);
    if (e != hipSuccess) return fail(HP_ERR_HIP, "local update launch: %s", hipGetErrorString(e));
    std::vector<int64_t> nv = v->V[newest];
    nv[v->id] += 1;
    v->V[slot] = nv;
    v->p = q;
    v->inflight -= 1;
    if (q % W == 0) v->push_due = true;
    return HP_OK;
}

extern "C" int hp_wsp_push_wave(hp_vw* v, hp_ps* ps) {
    if (!v || !ps) return fail(HP_ERR_ARG, "hp_wsp_push_wave: NULL argument");
    if (v->ps != ps) return fail(HP_ERR_ARG, "hp_wsp_push_wave: VW belongs to another server");
    if (!v->push_due)
        return fail(HP_ERR_STATE, "hp_wsp_push_wave: VW %d has no completed, unpushed wave", v->id);
    ps->timer.begin(2, ps->stream);
    hipError_t e = launch_wsp_push(ps->wg, v->ut, v->P, ps->stream);
    ps->timer.end(ps->stream);
    if (e != hipSuccess) return fail(HP_ERR_HIP, "push launch: %s", hipGetErrorString(e));
    ps->pushed[v->id] += 1;
    v->c = (int)(v->p / v->W);
    ps->clock[v->id] = v->c;
    ps->cg = *std::min_element(ps->clock.begin(), ps->clock.end());
    v->push_due = false;
    v->need_pull = true;
    return HP_OK;
}

extern "C" int hp_wsp_pull(hp_vw* v, hp_ps* ps) {
    if (!v || !ps) return fail(HP_ERR_ARG, "hp_wsp_pull: NULL argument");
    if (v->ps != ps) return fail(HP_ERR_ARG, "hp_wsp_pull: VW belongs to another server");
    if (!v->need_pull) return HP_OK;
    const int need = v->c - ps->D;
    if (v->g >= need) {            // the last pull still satisfies the bound
        v->need_pull = false;
        return HP_OK;
    }
    if (ps->cg < need) return HP_WOULD_BLOCK;
    const int slot = (int)((v->p - 1) % v->W);
    ps->timer.begin(3, ps->stream);
    hipError_t e = launch_wsp_copy(ps->wg, v->ring + (size_t)slot * v->stride, v->P, ps->stream);
    ps->timer.end(ps->stream);
    if (e != hipSuccess) return fail(HP_ERR_HIP, "pull launch: %s", hipGetErrorString(e));
    for (int n = 0; n < ps->N; ++n) v->V[slot][n] = (int64_t)v->W * ps->pushed[n];
    v->g = ps->cg;
    v->need_pull = false;
    return HP_OK;
}

extern "C" int hp_wsp_wave_end(hp_vw* v, hp_ps* ps, const float* grad, float lr) {
    if (!v || !ps || !grad) return fail(HP_ERR_ARG, "hp_wsp_wave_end: NULL argument");
    if (v->ps != ps) return fail(HP_ERR_ARG, "hp_wsp_wave_end: VW belongs to another server");
    if (v->inflight == 0)
        return fail(HP_ERR_STATE, "hp_wsp_wave_end: no minibatch was started (hp_wsp_weights)");
    if (v->push_due || v->need_pull)
        return fail(HP_ERR_STATE, "hp_wsp_wave_end: VW %d has an unsettled wave end", v->id);
    const int64_t q = v->p + 1;
    const int W = v->W;
    if (q % W != 0)
        return fail(HP_ERR_STATE, "hp_wsp_wave_end: minibatch %lld does not complete a wave",
                    (long long)q);
    const int slot = (int)((q - 1) % W);
    const int newest = (int)((q - 2 + W) % W);
    const int first = ((q - 1) % W) == 0;
    // the gate after the push, decided on the host before anything is enqueued
    const int c_new = (int)(q / W);
    int cg_new = c_new;
    for (int n = 0; n < ps->N; ++n)
        if (n != v->id) cg_new = std::min(cg_new, ps->clock[n]);
    const int need = c_new - ps->D;
    const bool satisfied = v->g >= need;
    const bool pull = !satisfied && cg_new >= need;
    StageTimer& tm = ps->timer;
    tm.begin(pull ? 4 : 5, ps->stream);
    hipError_t e = launch_wsp_wave_end(grad, v->ring + (size_t)newest * v->stride,
                                       v->ring + (size_t)slot * v->stride, v->ut,
                                       v->mu != 0.f ? v->vel : nullptr, ps->wg, v->P, lr, v->mu,
                                       first, pull ? 1 : 0, ps->stream);
    tm.end(ps->stream);
    if (e != hipSuccess) return fail(HP_ERR_HIP, "wave-end launch: %s", hipGetErrorString(e));
    // bookkeeping of the local update, the push and the gate, in that order
    std::vector<int64_t> nv = v->V[newest];
    nv[v->id] += 1;
    v->V[slot] = nv;
    v->p = q;
    v->inflight -= 1;
    ps->pushed[v->id] += 1;
    v->c = c_new;
    ps->clock[v->id] = c_new;
    ps->cg = *std::min_element(ps->clock.begin(), ps->clock.end());
    if (satisfied) return HP_OK;
    if (!pull) {
        v->need_pull = true;
        return HP_WOULD_BLOCK;
    }
    for (int n = 0; n < ps->N; ++n) v->V[slot][n] = (int64_t)W * ps->pushed[n];
    v->g = ps->cg;
    return HP_OK;
}

extern "C" int hp_wsp_state(const hp_vw* v, hp_wsp_state_t* out) {
    if (!v || !out) return fail(HP_ERR_ARG, "hp_wsp_state: NULL argument");
    out->p = v->p;
    out->W = v->W;
    out->c = v->c;
    out->g = v->g;
    out->push_due = v->push_due ? 1 : 0;
    out->gated = v->need_pull ? 1 : 0;
    out->next_slot = (int)((v->p + v->inflight) % v->W);
    out->in_flight = v->inflight;
    out->n_vw = v->ps ? v->ps->N : (int)v->V[0].size();
    return HP_OK;
}

extern "C" int hp_wsp_version(const hp_vw* v, int64_t* V) {
    if (!v || !V) return fail(HP_ERR_ARG, "hp_wsp_version: NULL argument");
    const std::vector<int64_t>& vv = v->V[(size_t)((v->p + v->inflight) % v->W)];
    for (size_t n = 0; n < vv.size(); ++n) V[n] = vv[n];
    return HP_OK;
}

extern "C" int hp_wsp_buffers(const hp_vw* v, const float** ring, size_t* slot_stride,
                              const float** utilde) {
    if (!v || !ring || !slot_stride || !utilde)
        return fail(HP_ERR_ARG, "hp_wsp_buffers: NULL argument");
    *ring = v->ring;
    *slot_stride = v->stride;
    *utilde = v->ut;
    return HP_OK;
}

extern "C" const char* hp_last_error(void) { return g_last_error.c_str(); }
