// Host engine behind the C ABI (include/ebrl.h): policy creation (seeded
// weights, packing, upload), the paged KV pool and its block allocator,
// per-call metadata, and the layer schedules of prefill, autoregressive
// action decode and flow-matching denoising.  Every step of the forward
// runs in the kernels of gemm.hip, attention.hip and misc.hip.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <map>
#include <mutex>
#include <numeric>
#include <string>
#include <vector>

#include "../../include/ebrl.h"
#include "../../include/ebrl_ops.h"
#include "kernels.h"
#include "weights.h"

using namespace ebrl;

namespace {

thread_local std::string g_create_error;

// CU count of every stream made by ebrl_stream_create_cu_masked (the bits set
// in its mask), read by the policies bound to it for the GEMM plan.
std::mutex g_stream_mu;
std::map<hipStream_t, int> g_stream_cus;

struct LayerW {
    void* qkv = nullptr;   // [(hq + 2 hkv) hd, d]: q rows, then k rows, then v rows
    void* o = nullptr;     // [d, hq hd]
    void* gu = nullptr;    // [2 mlp, d]: 32-row groups of 16 gate rows + 16 up rows
    void* down = nullptr;  // [d, mlp]
};

struct StackDims { int n = 0, d = 0, hq = 0, hkv = 0, hd = 0, mlp = 0; };

struct ProfRec { int cls; hipEvent_t a, b; double flop, bytes; };

// T: prefix length; noise_calls: the env's denoise calls that drew seeded noise
struct EnvSlot { int T = 0; std::vector<int> blocks; uint32_t noise_calls = 0; };

}  // namespace

struct ebrl_policy {
    ebrl_config cfg{};
    bool bf16 = true;
    size_t esz = 2;
    uint64_t seed = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    int dev_cus = 256;   // compute units of the device
    int cus = 256;       // ... that the bound stream may use
    std::string err;
    bool failed = false;

    // derived dims
    StackDims dec, vit, exp;
    int kpad = 0;          // padded patch length
    int patches_per_env = 0;
    int n_img = 0;         // decoder tokens from images per env
    int tail = 0;          // KV slots past the prefix (action tokens / chunk)
    int bt_stride = 0;     // blocks per env
    int max_pos = 0;

    // weights
    void *w_pe = nullptr, *e_lang = nullptr, *e_act = nullptr, *w_act = nullptr;
    void *vit_pos = nullptr, *w_proj = nullptr;
    void *w_ain = nullptr, *w_t1 = nullptr, *w_t2 = nullptr, *w_aout = nullptr;
    void *w_fin = nullptr, *w_fout = nullptr;   // world action model: frame latents in / out
    std::vector<LayerW> L_dec, L_vit, L_exp;

    // paged KV
    void* kv_pool = nullptr;
    int num_blocks = 0;
    size_t block_elems = 0;   // elements of one block in one layer
    std::vector<int> free_blocks;
    std::vector<EnvSlot> envs;
    std::vector<int> bt_host;
    int* bt_dev = nullptr;
    // ViT KV scratch (identity block table)
    void* vit_kv = nullptr;
    int* vit_bt = nullptr;
    int vit_bt_stride = 0;

    float* cos_tab = nullptr;
    float* sin_tab = nullptr;
    float* temb = nullptr;     // [n_steps, exp_d] time embeddings
    float* tvec = nullptr;     // [n_steps, exp_d] time-MLP outputs
    float* tmid = nullptr;

    // activations
    size_t rows_cap = 0;
    float* X = nullptr;        // residual stream
    void* Xn = nullptr;        // normed rows (act dtype)
    void* Qb = nullptr;
    void* Ob = nullptr;
    void* Hb = nullptr;
    void* patches = nullptr;
    float* Vx = nullptr;       // ViT residual stream
    float* h_pre = nullptr;    // [max_envs + 1, d] (the last row: the padding env)
    float* h_norm = nullptr;
    float* ws = nullptr;       // split-K workspace
    size_t ws_floats = 0;
    unsigned* counters = nullptr;  // split-K tile counters (zero between calls)
    float* lg = nullptr;           // action logits scratch [dec_cap][n_bins]
    unsigned* lg_counters = nullptr;
    // Decode calls run on a batch-size class (dec_class): rows past the
    // call's n are padding rows of env `pad_env` (an internal slot past the
    // caller's ids with a one-token zero prefix).  Outputs go to these
    // policy-owned buffers and are copied to the caller's after the graph.
    int dec_cap = 0;
    int pad_env = 0;
    int* dec_tok = nullptr;        // [dec_cap][n_action_tokens]
    float* dec_act = nullptr;
    float* dec_mar = nullptr;
    float* part = nullptr;     // decode attention partials
    size_t part_floats = 0;
    unsigned* attn_counters = nullptr;  // decode attention chunk counters [dec_cap][q_heads] (zero between calls)
    float* flow_x = nullptr;
    float* flow_v0 = nullptr;
    float* flow_f = nullptr;   // frame latents being denoised
    std::vector<int> last_flow_ids;

    // per-call metadata
    int* meta_dev = nullptr;
    int* meta_host = nullptr;
    size_t meta_cap = 0;       // ints
    hipEvent_t meta_ev = nullptr;
    bool meta_used = false;

    // profiling
    bool prof = false;
    int prof_mask = 0;
    std::vector<ProfRec> recs;
    std::vector<hipEvent_t> ev_pool;
    int64_t p_launch[EBRL_K_COUNT] = {};
    double p_ms[EBRL_K_COUNT] = {}, p_flop[EBRL_K_COUNT] = {}, p_bytes[EBRL_K_COUNT] = {};
    int cur_cls = -1;
    hipEvent_t cur_a = nullptr;

    // HIP graphs of whole decode / denoise calls, keyed by the call's batch
    // size class (decode) or batch size (denoise) and the bound stream's CU
    // count (which picks GEMM tile shapes) only: the per-call metadata
    // lives at fixed offsets of meta_dev and is refreshed by an async copy
    // before each launch, and inputs and outputs pass through policy-owned
    // buffers outside the graph, so new caller pointers never re-capture
    hipStream_t cap_stream = nullptr;
    std::map<std::vector<uint64_t>, hipGraphExec_t> graphs;

    std::vector<void*> allocs;
};

namespace {

// ------------------------------------------------------------- helpers --

int fail(ebrl_policy* p, int code, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
int fail(ebrl_policy* p, int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    if (p) {
        p->err = buf;
        if (code == EBRL_E_HIP) p->failed = true;
    } else {
        g_create_error = buf;
    }
    return code;
}

#define HIPCHK(p, call)                                                                        \
    do {                                                                                       \
        hipError_t e_ = (call);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail((p), e_ == hipErrorOutOfMemory ? EBRL_E_OOM : EBRL_E_HIP, "%s: %s (%s:%d)", \
                        #call, hipGetErrorString(e_), __FILE__, __LINE__);                    \
    } while (0)

int dev_alloc(ebrl_policy* p, void** out, size_t bytes) {
    *out = nullptr;
    if (bytes == 0) return EBRL_OK;
    hipError_t e = hipMalloc(out, bytes);
    if (e != hipSuccess) {
        *out = nullptr;
        (void)hipGetLastError();
        return fail(p, EBRL_E_OOM, "hipMalloc(%zu bytes) failed: %s", bytes, hipGetErrorString(e));
    }
    p->allocs.push_back(*out);
    return EBRL_OK;
}

template <typename T> int dev_alloc_t(ebrl_policy* p, T** out, size_t count) {
    return dev_alloc(p, reinterpret_cast<void**>(out), count * sizeof(T));
}

int check_launch(ebrl_policy* p) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(p, EBRL_E_HIP, "kernel launch: %s", hipGetErrorString(e));
    return EBRL_OK;
}

// ---------------------------------------------------------- profiling --

hipEvent_t get_event(ebrl_policy* p) {
    if (!p->ev_pool.empty()) {
        hipEvent_t e = p->ev_pool.back();
        p->ev_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    (void)hipEventCreate(&e);
    return e;
}

void prof_begin(ebrl_policy* p, int cls) {
    if (!p->prof || !(p->prof_mask & (1 << cls))) return;
    p->cur_cls = cls;
    p->cur_a = get_event(p);
    (void)hipEventRecord(p->cur_a, p->stream);
}

void prof_end(ebrl_policy* p, double flop, double bytes) {
    if (!p->prof || p->cur_cls < 0) return;
    hipEvent_t b = get_event(p);
    (void)hipEventRecord(b, p->stream);
    p->recs.push_back({p->cur_cls, p->cur_a, b, flop, bytes});
    p->cur_cls = -1;
}

void prof_collect(ebrl_policy* p) {
    if (p->recs.empty()) return;
    (void)hipStreamSynchronize(p->stream);
    for (auto& r : p->recs) {
        float ms = 0.f;
        (void)hipEventElapsedTime(&ms, r.a, r.b);
        p->p_launch[r.cls] += 1;
        p->p_ms[r.cls] += ms;
        p->p_flop[r.cls] += r.flop;
        p->p_bytes[r.cls] += r.bytes;
        p->ev_pool.push_back(r.a);
        p->ev_pool.push_back(r.b);
    }
    p->recs.clear();
}

// ------------------------------------------------------------ metadata --

struct Meta {
    std::vector<int> data;
    size_t add(const std::vector<int>& v) {
        size_t off = data.size();
        data.insert(data.end(), v.begin(), v.end());
        while (data.size() % 4) data.push_back(0);  // 16-byte alignment
        return off;
    }
};

// Copies the call's metadata (and the block table when `with_bt`) to the
// device on the bound stream; returns the device base pointer of `m`.
int upload_meta(ebrl_policy* p, const Meta& m, bool with_bt, int** dev) {
    const size_t n_meta = m.data.size();
    const size_t n_bt = with_bt ? p->bt_host.size() : 0;
    if (n_meta + n_bt > p->meta_cap)
        return fail(p, EBRL_E_INVALID, "call metadata (%zu ints) exceeds capacity %zu", n_meta + n_bt,
                    p->meta_cap);
    if (p->meta_used) HIPCHK(p, hipEventSynchronize(p->meta_ev));
    memcpy(p->meta_host, m.data.data(), n_meta * sizeof(int));
    if (n_bt) memcpy(p->meta_host + n_meta, p->bt_host.data(), n_bt * sizeof(int));
    if (n_meta)
        HIPCHK(p, hipMemcpyAsync(p->meta_dev, p->meta_host, n_meta * sizeof(int), hipMemcpyHostToDevice,
                                 p->stream));
    if (n_bt)
        HIPCHK(p, hipMemcpyAsync(p->bt_dev, p->meta_host + n_meta, n_bt * sizeof(int),
                                 hipMemcpyHostToDevice, p->stream));
    HIPCHK(p, hipEventRecord(p->meta_ev, p->stream));
    p->meta_used = true;
    *dev = p->meta_dev;
    return EBRL_OK;
}

// -------------------------------------------------------------- weights --

enum { TID_PATCH = 1, TID_ELANG, TID_EACT, TID_WACT, TID_VITPOS, TID_PROJ, TID_AIN, TID_T1, TID_T2,
       TID_AOUT, TID_FIN, TID_FOUT };
enum { SLOT_Q = 0, SLOT_K, SLOT_V, SLOT_O, SLOT_GATE, SLOT_UP, SLOT_DOWN };

// Where a logical tensor lives on the device.
struct Placement {
    void* buf = nullptr;     // device buffer holding it
    int buf_rows = 0;        // rows of that buffer
    int ld = 0;              // its row length (elements)
    int rows = 0, cols = 0;  // logical shape
    int kind = 0;            // 0 plain rows at row_off, 1 gate rows, 2 up rows,
                             // 3 rotary-paired rows inside heads of hd rows
    int row_off = 0;
    int hd = 0;
    bool ok = false;
    int dev_row(int i) const {
        if (kind == 1) return (i / 16) * 32 + (i % 16);
        if (kind == 2) return (i / 16) * 32 + 16 + (i % 16);
        if (kind == 3) {
            // head-local row e: first-half rows e < hd/2 and their rotation
            // partners e + hd/2 interleave in 16-row blocks
            const int h = i / hd, e = i % hd, half = hd / 2;
            const int pe = e < half ? (e / 16) * 32 + (e % 16) : ((e - half) / 16) * 32 + 16 + ((e - half) % 16);
            return row_off + h * hd + pe;
        }
        return row_off + i;
    }
};

Placement placement(const ebrl_policy* p, uint32_t tid) {
    Placement pl;
    const ebrl_config& c = p->cfg;
    auto plain = [&](void* buf, int rows, int cols, int ld) {
        pl.buf = buf; pl.buf_rows = rows; pl.ld = ld; pl.rows = rows; pl.cols = cols; pl.ok = buf != nullptr;
    };
    switch (tid) {
    case TID_PATCH: plain(p->w_pe, c.vit_layers ? c.vit_d : c.d, c.patch * c.patch * 3, p->kpad); return pl;
    case TID_ELANG: plain(p->e_lang, c.vocab, c.d, c.d); return pl;
    case TID_EACT: plain(p->e_act, c.n_bins, c.d, c.d); return pl;
    case TID_WACT: plain(p->w_act, c.n_bins, c.d, c.d); return pl;
    case TID_VITPOS: plain(p->vit_pos, p->patches_per_env, c.vit_d, c.vit_d); return pl;
    case TID_PROJ: plain(p->w_proj, c.d, c.vit_d, c.vit_d); return pl;
    case TID_AIN: plain(p->w_ain, c.exp_d, c.adim, c.adim); return pl;
    case TID_T1: plain(p->w_t1, c.exp_d, c.exp_d, c.exp_d); return pl;
    case TID_T2: plain(p->w_t2, c.exp_d, c.exp_d, c.exp_d); return pl;
    case TID_AOUT: plain(p->w_aout, c.adim, c.exp_d, c.exp_d); return pl;
    case TID_FIN: plain(p->w_fin, c.exp_d, c.frame_dim, c.frame_dim); return pl;
    case TID_FOUT: plain(p->w_fout, c.frame_dim, c.exp_d, c.exp_d); return pl;
    default: break;
    }
    const std::vector<LayerW>* layers = nullptr;
    const StackDims* sd = nullptr;
    uint32_t base = 0;
    if (tid >= 3000) { layers = &p->L_exp; sd = &p->exp; base = 3000; }
    else if (tid >= 2000) { layers = &p->L_vit; sd = &p->vit; base = 2000; }
    else if (tid >= 1000) { layers = &p->L_dec; sd = &p->dec; base = 1000; }
    else return pl;
    const int l = (int)((tid - base) / 16), slot = (int)((tid - base) % 16);
    if (l >= (int)layers->size()) return pl;
    const LayerW& w = (*layers)[l];
    const int qn = sd->hq * sd->hd, kn = sd->hkv * sd->hd, qkvn = qn + 2 * kn;
    switch (slot) {
    case SLOT_Q: plain(w.qkv, qn, sd->d, sd->d); pl.buf_rows = qkvn; pl.kind = 3; pl.hd = sd->hd; return pl;
    case SLOT_K: plain(w.qkv, kn, sd->d, sd->d); pl.buf_rows = qkvn; pl.row_off = qn; pl.kind = 3; pl.hd = sd->hd; return pl;
    case SLOT_V:
        plain(w.qkv, kn, sd->d, sd->d); pl.buf_rows = qkvn; pl.row_off = qn + kn; pl.kind = 3; pl.hd = sd->hd;
        return pl;
    case SLOT_O: plain(w.o, sd->d, qn, qn); return pl;
    case SLOT_GATE: plain(w.gu, sd->mlp, sd->d, sd->d); pl.buf_rows = 2 * sd->mlp; pl.kind = 1; return pl;
    case SLOT_UP: plain(w.gu, sd->mlp, sd->d, sd->d); pl.buf_rows = 2 * sd->mlp; pl.kind = 2; return pl;
    case SLOT_DOWN: plain(w.down, sd->d, sd->mlp, sd->mlp); return pl;
    default: return pl;
    }
}

// Scatter a logical [rows, cols] tensor into a host image of its device buffer.
void scatter_rows(const Placement& pl, const void* logical, char* image, size_t esz) {
    for (int i = 0; i < pl.rows; ++i)
        memcpy(image + (size_t)pl.dev_row(i) * pl.ld * esz, (const char*)logical + (size_t)i * pl.cols * esz,
               (size_t)pl.cols * esz);
}

void gather_rows(const Placement& pl, const char* image, void* logical, size_t esz) {
    for (int i = 0; i < pl.rows; ++i)
        memcpy((char*)logical + (size_t)i * pl.cols * esz, image + (size_t)pl.dev_row(i) * pl.ld * esz,
               (size_t)pl.cols * esz);
}

// Generate the tensors sharing one device buffer and upload it.
int fill_buffer(ebrl_policy* p, const std::vector<uint32_t>& tids) {
    if (tids.empty()) return EBRL_OK;
    const Placement first = placement(p, tids[0]);
    if (!first.ok) return fail(p, EBRL_E_INVALID, "internal: no placement for tensor %u", tids[0]);
    const size_t bytes = (size_t)first.buf_rows * first.ld * p->esz;
    std::vector<char> image(bytes, 0);
    std::vector<char> logical;
    for (uint32_t t : tids) {
        const Placement pl = placement(p, t);
        logical.resize((size_t)pl.rows * pl.cols * p->esz);
        generate_weight(p->seed, t, (int64_t)pl.rows * pl.cols, p->cfg.init_std, p->bf16, logical.data());
        scatter_rows(pl, logical.data(), image.data(), p->esz);
    }
    HIPCHK(p, hipMemcpy(first.buf, image.data(), bytes, hipMemcpyHostToDevice));
    return EBRL_OK;
}

int alloc_stack(ebrl_policy* p, std::vector<LayerW>& Ls, const StackDims& s) {
    Ls.resize(s.n);
    const size_t qkvn = (size_t)(s.hq + 2 * s.hkv) * s.hd;
    for (auto& w : Ls) {
        int rc;
        if ((rc = dev_alloc(p, &w.qkv, qkvn * s.d * p->esz))) return rc;
        if ((rc = dev_alloc(p, &w.o, (size_t)s.d * s.hq * s.hd * p->esz))) return rc;
        if ((rc = dev_alloc(p, &w.gu, (size_t)2 * s.mlp * s.d * p->esz))) return rc;
        if ((rc = dev_alloc(p, &w.down, (size_t)s.d * s.mlp * p->esz))) return rc;
    }
    return EBRL_OK;
}

int fill_stack(ebrl_policy* p, uint32_t base, int n) {
    for (int l = 0; l < n; ++l) {
        const uint32_t b = base + 16u * l;
        int rc;
        if ((rc = fill_buffer(p, {b + SLOT_Q, b + SLOT_K, b + SLOT_V}))) return rc;
        if ((rc = fill_buffer(p, {b + SLOT_O}))) return rc;
        if ((rc = fill_buffer(p, {b + SLOT_GATE, b + SLOT_UP}))) return rc;
        if ((rc = fill_buffer(p, {b + SLOT_DOWN}))) return rc;
    }
    return EBRL_OK;
}

// -------------------------------------------------------------- config --

int validate(const ebrl_config& c, std::string& why) {
    auto bad = [&](const char* m) { why = m; return EBRL_E_INVALID; };
    if (c.dtype != EBRL_DTYPE_FP32 && c.dtype != EBRL_DTYPE_BF16) return bad("dtype");
    if (c.layers < 1 || c.d < 64 || c.d % 64) return bad("decoder width must be a positive multiple of 64");
    if (c.head_dim != 64 && c.head_dim != 128) return bad("head_dim must be 64 or 128");
    if (c.q_heads < 1 || c.kv_heads < 1 || c.q_heads % c.kv_heads) return bad("heads");
    if (c.mlp < 16 || c.mlp % 16) return bad("mlp must be a multiple of 16");
    if (c.vocab < 1 || c.n_lang < 0) return bad("vocab / n_lang");
    if (c.n_cams < 0 || (c.n_cams > 0 && (c.patch < 1 || c.img < c.patch || c.img % c.patch)))
        return bad("image / patch");
    if (c.vit_layers) {
        if (c.vit_d < 64 || c.vit_d % 64 || c.vit_heads < 1 || c.vit_d % c.vit_heads) return bad("vit dims");
        const int vhd = c.vit_d / c.vit_heads;
        if (vhd != 64 && vhd != 128) return bad("vit head dim must be 64 or 128");
        if (c.vit_mlp < 16 || c.vit_mlp % 16) return bad("vit mlp");
    }
    if (c.action_logits && (c.n_bins < 2 || c.n_action_tokens < 1)) return bad("action head");
    if (c.exp_layers) {
        if (c.exp_d < 64 || c.exp_d % 64 || c.exp_mlp % 16 || c.exp_mlp < 16) return bad("expert dims");
        if (c.exp_heads != c.kv_heads) return bad("expert heads must equal backbone kv heads");
        if (c.chunk < 1 || c.adim < 1 || c.adim > 64 || c.n_steps < 1) return bad("flow chunk / action dims / steps");
    }
    if (c.frame_tokens < 0 || (c.frame_tokens > 0 && (!c.exp_layers || c.frame_dim < 1 || c.frame_dim > 64)))
        return bad("frame tokens need an expert and 1 <= frame_dim <= 64");
    if (!c.action_logits && !c.exp_layers) return bad("no action head and no expert");
    if (c.max_envs < 1 || c.max_seq < 1) return bad("capacity");
    if (!(c.init_std > 0.0)) return bad("init_std");
    {
        // the bf16 attention kernels stage a sequence's block table in LDS
        const int tail =
            std::max(c.action_logits ? c.n_action_tokens - 1 : 0, c.exp_layers ? c.chunk + c.frame_tokens : 0);
        const int blocks = (c.max_seq + tail + KV_BLOCK - 1) / KV_BLOCK;
        const int vit_blocks =
            c.n_cams ? (c.n_cams * (c.img / c.patch) * (c.img / c.patch) + KV_BLOCK - 1) / KV_BLOCK : 0;
        if (c.dtype == EBRL_DTYPE_BF16 && std::max(blocks, vit_blocks) > ATTN_BT_MAX)
            return bad("sequence too long for the bf16 attention kernels (4096 tokens per sequence)");
    }
    return EBRL_OK;
}

// --------------------------------------------------------- GEMM launch --

int run_gemm(ebrl_policy* p, GemmArgs a, bool split_ok = false) {
    a.bf16 = p->bf16;
    a.split_ok = split_ok;
    a.ws = p->ws;
    a.ws_floats = p->ws_floats;
    a.counters = p->counters;
    a.cus = p->cus;
    const int cls = a.M >= 256 ? EBRL_K_GEMM : EBRL_K_GEMM_SKINNY;
    prof_begin(p, cls);
    ebrl::gemm(a, p->stream);
    const double flop = 2.0 * a.M * (double)a.N * a.K;
    const double outb = (a.epi == EPI_SWIGLU ? (double)a.M * a.N / 2 : (double)a.M * a.N) *
                        (a.epi == EPI_SWIGLU || a.epi == EPI_QKV ? p->esz : 4);
    prof_end(p, flop, ((double)a.M * a.K + (double)a.N * a.K) * p->esz + outb);
    return EBRL_OK;
}

// One pre-norm transformer block over `rows` rows of residual stream R.
struct BlockCall {
    float* R = nullptr; int rows = 0;
    const StackDims* sd = nullptr;
    const LayerW* w = nullptr;
    PagedKV kv;
    const int* seq_env = nullptr;
    const int* row_seq = nullptr;
    const int* row_pos = nullptr;
    bool use_rope = true;
    // attention
    bool decode = false;
    double attn_flop = 0, attn_bytes = 0;  // algorithmic work of the attention launch
    AttnPrefillArgs pre;
    AttnDecodeArgs dec;
};

// Decode steps of bf16 policies fold each pre-norm into the projection that
// follows it: the residual stream's producers (embedding, O and down
// projections) also store the rows in bf16, and the QKV and gate/up decode
// GEMMs scale their output rows by the RMSNorm factor of those rows.
bool fold_decode_norm(const ebrl_policy* p, const StackDims& s, int rows) {
    const int qkvn = (s.hq + 2 * s.hkv) * s.hd;
    return p->bf16 && gemm_row_norm_ok(true, rows, qkvn, s.d, p->ws_floats) &&
           gemm_row_norm_ok(true, rows, 2 * s.mlp, s.d, p->ws_floats);
}

int run_block(ebrl_policy* p, BlockCall& b) {
    const StackDims& s = *b.sd;
    const int qn = s.hq * s.hd, qkvn = (s.hq + 2 * s.hkv) * s.hd;
    const bool fold = b.decode && fold_decode_norm(p, s, b.rows);
    if (!fold) {
        prof_begin(p, EBRL_K_OTHER);
        rmsnorm_rows(p->bf16, b.R, s.d, nullptr, p->Xn, s.d, b.rows, s.d, 1e-6f, p->stream);
        prof_end(p, 0, (double)b.rows * s.d * (4 + p->esz));
    }
    // fused QKV projection: rotary embedding of Q and K and the paged K/V
    // write happen in the GEMM epilogue
    RopeKVArgs r;
    r.bf16 = p->bf16; r.M = b.rows; r.q_heads = s.hq;
    r.Q = p->Qb; r.ldq = qn; r.kv = b.kv; r.seq_env = b.seq_env; r.row_seq = b.row_seq;
    r.row_pos = b.row_pos; r.cos_tab = p->cos_tab; r.sin_tab = p->sin_tab; r.use_rope = b.use_rope;
    GemmArgs g;
    g.A = p->Xn; g.lda = s.d; g.B = b.w->qkv; g.ldb = s.d; g.M = b.rows; g.N = qkvn; g.K = s.d;
    g.epi = EPI_QKV; g.rope = &r; g.row_norm = fold;
    run_gemm(p, g, b.decode);
    if (b.decode) {
        b.dec.bf16 = p->bf16; b.dec.Q = p->Qb; b.dec.ldq = qn; b.dec.O = p->Ob; b.dec.ldo = qn;
        b.dec.q_heads = s.hq; b.dec.kv = b.kv; b.dec.part = p->part; b.dec.counters = p->attn_counters;
        prof_begin(p, EBRL_K_ATTN_DECODE);
        attn_decode(b.dec, p->stream);
        prof_end(p, b.attn_flop, b.attn_bytes);
    } else {
        b.pre.bf16 = p->bf16; b.pre.Q = p->Qb; b.pre.ldq = qn; b.pre.O = p->Ob; b.pre.ldo = qn;
        b.pre.q_heads = s.hq; b.pre.kv = b.kv;
        prof_begin(p, EBRL_K_ATTN_PREFILL);
        attn_prefill(b.pre, p->stream);
        prof_end(p, b.attn_flop, b.attn_bytes);
    }
    g = GemmArgs();
    g.A = p->Ob; g.lda = qn; g.B = b.w->o; g.ldb = qn; g.M = b.rows; g.N = s.d; g.K = qn;
    g.epi = EPI_RESID; g.C = b.R; g.ldc = s.d;
    if (fold) { g.xb = p->Xn; g.ldxb = s.d; }
    run_gemm(p, g, b.decode);
    if (!fold) {
        prof_begin(p, EBRL_K_OTHER);
        rmsnorm_rows(p->bf16, b.R, s.d, nullptr, p->Xn, s.d, b.rows, s.d, 1e-6f, p->stream);
        prof_end(p, 0, (double)b.rows * s.d * (4 + p->esz));
    }
    g = GemmArgs();
    g.A = p->Xn; g.lda = s.d; g.B = b.w->gu; g.ldb = s.d; g.M = b.rows; g.N = 2 * s.mlp; g.K = s.d;
    g.epi = EPI_SWIGLU; g.C = p->Hb; g.ldc = s.mlp; g.row_norm = fold;
    run_gemm(p, g, b.decode);
    g = GemmArgs();
    g.A = p->Hb; g.lda = s.mlp; g.B = b.w->down; g.ldb = s.mlp; g.M = b.rows; g.N = s.d; g.K = s.mlp;
    g.epi = EPI_RESID; g.C = b.R; g.ldc = s.d;
    if (fold) { g.xb = p->Xn; g.ldxb = s.d; }
    run_gemm(p, g, b.decode);
    return EBRL_OK;
}

int check_ready(ebrl_policy* p) {
    if (!p) return EBRL_E_INVALID;
    if (p->failed) return EBRL_E_HIP;
    int dev = -1;
    if (hipGetDevice(&dev) == hipSuccess && dev != p->device) HIPCHK(p, hipSetDevice(p->device));
    return EBRL_OK;
}

int check_ids(ebrl_policy* p, const int32_t* ids, int n, bool need_prefix) {
    if (n < 0 || n > p->cfg.max_envs) return fail(p, EBRL_E_INVALID, "n = %d outside [0, %d]", n, p->cfg.max_envs);
    if (n > 0 && !ids) return fail(p, EBRL_E_INVALID, "env_ids is NULL");
    std::vector<char> seen(p->cfg.max_envs, 0);
    for (int i = 0; i < n; ++i) {
        const int e = ids[i];
        if (e < 0 || e >= p->cfg.max_envs) return fail(p, EBRL_E_INVALID, "env id %d out of range", e);
        if (seen[e]) return fail(p, EBRL_E_INVALID, "duplicate env id %d", e);
        seen[e] = 1;
        if (need_prefix && p->envs[e].T <= 0)
            return fail(p, EBRL_E_STATE, "env %d has no prefix (call ebrl_prefill first)", e);
    }
    return EBRL_OK;
}

PagedKV dec_kv(const ebrl_policy* p, int layer) {
    PagedKV k;
    k.base = (char*)p->kv_pool + (size_t)layer * p->num_blocks * p->block_elems * p->esz;
    k.block_table = p->bt_dev;
    k.bt_stride = p->bt_stride;
    k.kv_heads = p->cfg.kv_heads;
    k.head_dim = p->cfg.head_dim;
    return k;
}

// Enqueue `body` on the bound stream as a cached HIP graph, unless per-kernel
// timing is on for a kernel class the body launches (`classes`, a bit mask):
// then it runs eagerly so that every launch can be bracketed by events.
// `body` launches kernels on p->stream only.
int run_graph(ebrl_policy* p, const std::vector<uint64_t>& key, int classes, const std::function<int()>& body) {
    if (p->prof && (p->prof_mask & classes)) return body();
    auto it = p->graphs.find(key);
    if (it == p->graphs.end()) {
        if (p->graphs.size() >= 512) {
            HIPCHK(p, hipStreamSynchronize(p->stream));
            for (auto& kv : p->graphs) (void)hipGraphExecDestroy(kv.second);
            p->graphs.clear();
        }
        hipStream_t bound = p->stream;
        p->stream = p->cap_stream;
        HIPCHK(p, hipStreamBeginCapture(p->cap_stream, hipStreamCaptureModeRelaxed));
        int rc = body();
        hipGraph_t graph = nullptr;
        hipError_t e = hipStreamEndCapture(p->cap_stream, &graph);
        p->stream = bound;
        if (rc) {
            if (graph) (void)hipGraphDestroy(graph);
            return rc;
        }
        if (e != hipSuccess) return fail(p, EBRL_E_HIP, "graph capture: %s", hipGetErrorString(e));
        hipGraphExec_t exec = nullptr;
        e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
        (void)hipGraphDestroy(graph);
        if (e != hipSuccess) return fail(p, EBRL_E_HIP, "graph instantiate: %s", hipGetErrorString(e));
        it = p->graphs.emplace(key, exec).first;
    }
    HIPCHK(p, hipGraphLaunch(it->second, p->stream));
    return EBRL_OK;
}

// Flow-matching denoising of each env's token block -- frame_tokens
// future-frame latents (world action model only), then the action chunk --
// by the expert, attending to the env's backbone cache and, without a mask,
// to the block itself; Euler steps on both modalities at once.
int denoise(ebrl_policy* p, const int32_t* env_ids, int32_t n, const float* fnoise, const float* anoise,
            float* fout, float* aout) {
    const ebrl_config& c = p->cfg;
    int rc;
    if ((rc = check_ids(p, env_ids, n, true))) return rc;
    if (n == 0) return EBRL_OK;
    if (!aout) return fail(p, EBRL_E_INVALID, "out_actions is NULL");
    const int F = c.frame_tokens, S = F + c.chunk;
    // NULL noise: drawn on the device from the policy seed, the env id and
    // the env's count of such calls (frames on their own stream)
    const bool seeded = !anoise || (F && !fnoise);
    const int rows = n * S, arows = n * c.chunk, frows = n * F;
    std::vector<int> seq_env(env_ids, env_ids + n), q_off(n), q_len(n, S), q_pos0(n), kv_len(n),
        row_seq(rows), row_pos(rows), tseq, tq0, calls(n);
    for (int i = 0; i < n; ++i) {
        const int T = p->envs[env_ids[i]].T;
        calls[i] = (int)p->envs[env_ids[i]].noise_calls;
        q_off[i] = i * S;
        q_pos0[i] = T;
        kv_len[i] = T + S;
        for (int j = 0; j < S; ++j) { row_seq[i * S + j] = i; row_pos[i * S + j] = T + j; }
        for (int q0 = 0; q0 < S; q0 += ATTN_Q_TILE) { tseq.push_back(i); tq0.push_back(q0); }
    }
    Meta m;
    const size_t o_env = m.add(seq_env), o_off = m.add(q_off), o_len = m.add(q_len), o_pos0 = m.add(q_pos0),
                 o_kvl = m.add(kv_len), o_rseq = m.add(row_seq), o_rpos = m.add(row_pos), o_tseq = m.add(tseq),
                 o_tq0 = m.add(tq0), o_calls = m.add(calls);
    int* md = nullptr;
    if ((rc = upload_meta(p, m, false, &md))) return rc;
    // caller noise enters and the result leaves through the policy's own
    // buffers outside the graph, so the graph never holds a caller pointer
    prof_begin(p, EBRL_K_OTHER);
    if (anoise) copy_f32(anoise, p->flow_x, (size_t)arows * c.adim, p->stream);
    if (F && fnoise) copy_f32(fnoise, p->flow_f, (size_t)frows * c.frame_dim, p->stream);
    prof_end(p, 0, 0);
    auto body = [&]() -> int {
        // time-MLP outputs for the fixed tau schedule
        prof_begin(p, EBRL_K_OTHER);
        small_linear(p->bf16, p->temb, c.n_steps, c.exp_d, p->w_t1, c.exp_d, p->tmid, false, p->stream);
        small_linear(p->bf16, p->tmid, c.n_steps, c.exp_d, p->w_t2, c.exp_d, p->tvec, true, p->stream);
        if (!anoise)
            normal_noise(p->flow_x, n, c.chunk * c.adim, md + o_env, md + o_calls, p->seed, EBRL_NOISE_STREAM_ACTIONS,
                         p->stream);
        if (F && !fnoise)
            normal_noise(p->flow_f, n, F * c.frame_dim, md + o_env, md + o_calls, p->seed, EBRL_NOISE_STREAM_FRAMES,
                         p->stream);
        prof_end(p, 0, 0);
        for (int k = 0; k < c.n_steps; ++k) {
            const float* tv = p->tvec + (size_t)k * c.exp_d;
            prof_begin(p, EBRL_K_OTHER);
            if (F) flow_in(p->bf16, p->flow_f, frows, c.frame_dim, p->w_fin, tv, c.exp_d, p->X, c.exp_d, F, S, 0,
                           p->stream);
            flow_in(p->bf16, p->flow_x, arows, c.adim, p->w_ain, tv, c.exp_d, p->X, c.exp_d, c.chunk, S, F,
                    p->stream);
            prof_end(p, 0, 0);
            for (int l = 0; l < c.exp_layers; ++l) {
                BlockCall b;
                b.R = p->X; b.rows = rows; b.sd = &p->exp; b.w = &p->L_exp[l]; b.kv = dec_kv(p, l);
                b.seq_env = md + o_env; b.row_seq = md + o_rseq; b.row_pos = md + o_rpos;
                b.pre.seq_env = md + o_env; b.pre.q_off = md + o_off; b.pre.q_len = md + o_len;
                b.pre.q_pos0 = md + o_pos0; b.pre.kv_len = md + o_kvl; b.pre.tile_seq = md + o_tseq;
                b.pre.tile_q0 = md + o_tq0; b.pre.n_tiles = (int)tseq.size(); b.pre.causal = false;
                b.pre.max_kv_len = c.max_seq + S;   // the graph may serve longer prefixes later
                b.attn_flop = 0;
                // algorithmic bytes: Q read and O written once, every K/V row read once
                b.attn_bytes = 2.0 * n * S * p->exp.hq * c.head_dim * p->esz;
                for (int i = 0; i < n; ++i) {
                    b.attn_flop += 4.0 * c.head_dim * p->exp.hq * (double)S * kv_len[i];
                    b.attn_bytes += 2.0 * kv_len[i] * p->exp.hkv * c.head_dim * p->esz;
                }
                int rc2 = run_block(p, b);
                if (rc2) return rc2;
            }
            prof_begin(p, EBRL_K_OTHER);
            if (F) flow_out(p->bf16, p->X, c.exp_d, frows, c.exp_d, p->w_fout, c.frame_dim, 1e-6f, (float)c.n_steps,
                            p->flow_f, nullptr, F, S, 0, p->stream);
            flow_out(p->bf16, p->X, c.exp_d, arows, c.exp_d, p->w_aout, c.adim, 1e-6f, (float)c.n_steps, p->flow_x,
                     k == 0 ? p->flow_v0 : nullptr, c.chunk, S, F, p->stream);
            prof_end(p, 0, 0);
        }
        return check_launch(p);
    };
    // graph per (batch size, which noises are drawn on the device); the key
    // holds no caller pointer and no prefix length (the attention reads each
    // sequence's length from the metadata)
    const std::vector<uint64_t> key = {2, (uint64_t)n, (uint64_t)(anoise ? 1 : 0), (uint64_t)(fnoise ? 1 : 0),
                                       (uint64_t)p->cus};
    const int inside = (1 << EBRL_K_GEMM) | (1 << EBRL_K_GEMM_SKINNY) | (1 << EBRL_K_ATTN_PREFILL) |
                       (1 << EBRL_K_OTHER);
    if ((rc = run_graph(p, key, inside, body))) return rc;
    prof_begin(p, EBRL_K_OTHER);
    copy_f32(p->flow_x, aout, (size_t)arows * c.adim, p->stream);
    if (F) copy_f32(p->flow_f, fout, (size_t)frows * c.frame_dim, p->stream);
    prof_end(p, 0, 0);
    if (seeded)
        for (int i = 0; i < n; ++i) ++p->envs[env_ids[i]].noise_calls;
    p->last_flow_ids.assign(env_ids, env_ids + n);
    return check_launch(p);
}

}  // namespace

// =================================================================== ABI ==

extern "C" {

int ebrl_config_preset(int32_t preset, ebrl_config* out) {
    if (!out) return EBRL_E_INVALID;
    ebrl_config c;
    memset(&c, 0, sizeof(c));
    c.init_std = 0.02;
    c.action_logits = 1;
    c.n_action_tokens = 7;
    c.n_bins = 256;
    switch (preset) {
    case 1:  // tiny fp32 VLA
        c.dtype = EBRL_DTYPE_FP32; c.n_cams = 1; c.img = 64; c.patch = 16;
        c.layers = 2; c.d = 256; c.q_heads = 4; c.kv_heads = 4; c.head_dim = 64; c.mlp = 1024;
        c.vocab = 1024; c.n_lang = 8; c.max_envs = 8; c.max_seq = 24;
        break;
    case 2:  // small bf16 VLA
        c.dtype = EBRL_DTYPE_BF16; c.n_cams = 2; c.img = 224; c.patch = 16;
        c.layers = 12; c.d = 1024; c.q_heads = 16; c.kv_heads = 16; c.head_dim = 64; c.mlp = 4096;
        c.vocab = 32000; c.n_lang = 32; c.max_envs = 64; c.max_seq = 424;
        break;
    case 3:  // 7B-class bf16 VLA with ViT
        c.dtype = EBRL_DTYPE_BF16; c.n_cams = 1; c.img = 224; c.patch = 14;
        c.vit_layers = 24; c.vit_d = 1024; c.vit_heads = 16; c.vit_mlp = 4096;
        c.layers = 32; c.d = 4096; c.q_heads = 32; c.kv_heads = 32; c.head_dim = 128; c.mlp = 11008;
        c.vocab = 32000; c.n_lang = 32; c.max_envs = 32; c.max_seq = 288;
        break;
    case 4:  // flow-matching expert on a GQA backbone
    case 5:  // world action model: the same, also denoising latent future frames
        c.dtype = EBRL_DTYPE_BF16; c.n_cams = 3; c.img = 224; c.patch = 16;
        c.layers = 18; c.d = 2048; c.q_heads = 16; c.kv_heads = 8; c.head_dim = 128; c.mlp = 8192;
        c.vocab = 32000; c.n_lang = 12; c.action_logits = 0;
        c.exp_layers = 18; c.exp_d = 1024; c.exp_heads = 8; c.exp_mlp = 4096;
        c.chunk = 50; c.adim = 7; c.n_steps = 10; c.max_envs = 64; c.max_seq = 600;
        if (preset == 5) { c.frame_tokens = 98; c.frame_dim = 32; }
        break;
    default:
        return EBRL_E_INVALID;
    }
    *out = c;
    return EBRL_OK;
}

const char* ebrl_last_error(const ebrl_policy* p) {
    return p ? p->err.c_str() : g_create_error.c_str();
}

void ebrl_policy_destroy(ebrl_policy* p) {
    if (!p) return;
    (void)hipSetDevice(p->device);
    (void)hipStreamSynchronize(p->stream);
    for (auto& r : p->recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
    for (auto e : p->ev_pool) (void)hipEventDestroy(e);
    for (auto& kv : p->graphs) (void)hipGraphExecDestroy(kv.second);
    if (p->cap_stream) (void)hipStreamDestroy(p->cap_stream);
    if (p->meta_ev) (void)hipEventDestroy(p->meta_ev);
    if (p->meta_host) (void)hipHostFree(p->meta_host);
    for (void* a : p->allocs) (void)hipFree(a);
    delete p;
}

int ebrl_policy_create(const ebrl_config* config, uint64_t seed, ebrl_policy** out) {
    if (!out) return EBRL_E_INVALID;
    *out = nullptr;
    g_create_error.clear();
    if (!config) return fail(nullptr, EBRL_E_INVALID, "config is NULL");
    std::string why;
    if (validate(*config, why) != EBRL_OK) return fail(nullptr, EBRL_E_INVALID, "invalid config: %s", why.c_str());

    ebrl_policy* p = new ebrl_policy();
    p->cfg = *config;
    const ebrl_config& c = p->cfg;
    p->bf16 = c.dtype == EBRL_DTYPE_BF16;
    p->esz = p->bf16 ? 2 : 4;
    p->seed = seed;
    if (hipGetDevice(&p->device) != hipSuccess) {
        delete p;
        return fail(nullptr, EBRL_E_HIP, "no HIP device");
    }
    int ncu = 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, p->device) == hipSuccess && ncu > 0)
        p->dev_cus = p->cus = ncu;
    auto bail = [&](int rc) {
        g_create_error = p->err;
        ebrl_policy_destroy(p);
        return rc;
    };
    int rc;

    p->dec = {c.layers, c.d, c.q_heads, c.kv_heads, c.head_dim, c.mlp};
    if (c.vit_layers) p->vit = {c.vit_layers, c.vit_d, c.vit_heads, c.vit_heads, c.vit_d / c.vit_heads, c.vit_mlp};
    if (c.exp_layers) p->exp = {c.exp_layers, c.exp_d, c.exp_heads, c.exp_heads, c.head_dim, c.exp_mlp};
    const int pdim = c.patch * c.patch * 3;
    p->kpad = (pdim + 63) / 64 * 64;
    p->patches_per_env = c.n_cams ? c.n_cams * (c.img / c.patch) * (c.img / c.patch) : 0;
    p->n_img = p->patches_per_env;
    p->tail = std::max(c.action_logits ? c.n_action_tokens - 1 : 0, c.exp_layers ? c.chunk + c.frame_tokens : 0);
    p->bt_stride = (c.max_seq + p->tail + KV_BLOCK - 1) / KV_BLOCK;
    p->max_pos = c.max_seq + p->tail + 1;

    // ---- weights
    const int pe_out = c.vit_layers ? c.vit_d : c.d;
    if (c.n_cams && (rc = dev_alloc(p, &p->w_pe, (size_t)pe_out * p->kpad * p->esz))) return bail(rc);
    if ((rc = dev_alloc(p, &p->e_lang, (size_t)c.vocab * c.d * p->esz))) return bail(rc);
    if (c.action_logits) {
        if ((rc = dev_alloc(p, &p->e_act, (size_t)c.n_bins * c.d * p->esz))) return bail(rc);
        if ((rc = dev_alloc(p, &p->w_act, (size_t)c.n_bins * c.d * p->esz))) return bail(rc);
    }
    if (c.vit_layers) {
        if ((rc = dev_alloc(p, &p->vit_pos, (size_t)p->patches_per_env * c.vit_d * p->esz))) return bail(rc);
        if ((rc = dev_alloc(p, &p->w_proj, (size_t)c.d * c.vit_d * p->esz))) return bail(rc);
        if ((rc = alloc_stack(p, p->L_vit, p->vit))) return bail(rc);
    }
    if ((rc = alloc_stack(p, p->L_dec, p->dec))) return bail(rc);
    if (c.exp_layers) {
        if ((rc = dev_alloc(p, &p->w_ain, (size_t)c.exp_d * c.adim * p->esz))) return bail(rc);
        if ((rc = dev_alloc(p, &p->w_t1, (size_t)c.exp_d * c.exp_d * p->esz))) return bail(rc);
        if ((rc = dev_alloc(p, &p->w_t2, (size_t)c.exp_d * c.exp_d * p->esz))) return bail(rc);
        if ((rc = dev_alloc(p, &p->w_aout, (size_t)c.adim * c.exp_d * p->esz))) return bail(rc);
        if (c.frame_tokens) {
            if ((rc = dev_alloc(p, &p->w_fin, (size_t)c.exp_d * c.frame_dim * p->esz))) return bail(rc);
            if ((rc = dev_alloc(p, &p->w_fout, (size_t)c.frame_dim * c.exp_d * p->esz))) return bail(rc);
        }
        if ((rc = alloc_stack(p, p->L_exp, p->exp))) return bail(rc);
    }
    if (c.n_cams && (rc = fill_buffer(p, {TID_PATCH}))) return bail(rc);
    if ((rc = fill_buffer(p, {TID_ELANG}))) return bail(rc);
    if (c.action_logits) {
        if ((rc = fill_buffer(p, {TID_EACT}))) return bail(rc);
        if ((rc = fill_buffer(p, {TID_WACT}))) return bail(rc);
    }
    if (c.vit_layers) {
        if ((rc = fill_buffer(p, {TID_VITPOS}))) return bail(rc);
        if ((rc = fill_buffer(p, {TID_PROJ}))) return bail(rc);
        if ((rc = fill_stack(p, 2000, c.vit_layers))) return bail(rc);
    }
    if ((rc = fill_stack(p, 1000, c.layers))) return bail(rc);
    if (c.exp_layers) {
        for (uint32_t t : {TID_AIN, TID_T1, TID_T2, TID_AOUT})
            if ((rc = fill_buffer(p, {t}))) return bail(rc);
        if (c.frame_tokens)
            for (uint32_t t : {TID_FIN, TID_FOUT})
                if ((rc = fill_buffer(p, {t}))) return bail(rc);
        if ((rc = fill_stack(p, 3000, c.exp_layers))) return bail(rc);
    }

    // ---- paged KV pool
    p->block_elems = (size_t)2 * c.kv_heads * KV_BLOCK * c.head_dim;
    const size_t block_bytes_all = p->block_elems * p->esz * c.layers;
    int64_t budget = c.kv_budget_bytes;
    if (budget <= 0) budget = (int64_t)block_bytes_all * p->bt_stride * c.max_envs;
    const int budget_blocks = (int)(budget / (int64_t)block_bytes_all);
    if (budget_blocks < p->bt_stride) {
        fail(p, EBRL_E_INVALID, "kv_budget_bytes holds %d blocks, one env needs %d", budget_blocks, p->bt_stride);
        return bail(EBRL_E_INVALID);
    }
    // the padding env of decode size classes: a one-token prefix of zeros
    // plus its action-token slots, in blocks of its own outside the budget
    p->pad_env = c.max_envs;
    const int pad_blocks = (1 + p->tail + KV_BLOCK - 1) / KV_BLOCK;
    p->num_blocks = budget_blocks + pad_blocks;
    if ((rc = dev_alloc(p, &p->kv_pool, (size_t)p->num_blocks * block_bytes_all))) return bail(rc);
    p->free_blocks.resize(budget_blocks);
    for (int b = 0; b < budget_blocks; ++b) p->free_blocks[b] = budget_blocks - 1 - b;
    p->envs.assign(c.max_envs + 1, EnvSlot());
    p->bt_host.assign((size_t)(c.max_envs + 1) * p->bt_stride, 0);
    {
        EnvSlot& pad = p->envs[p->pad_env];
        pad.T = 1;
        for (int b = 0; b < pad_blocks; ++b) {
            pad.blocks.push_back(budget_blocks + b);
            p->bt_host[(size_t)p->pad_env * p->bt_stride + b] = budget_blocks + b;
        }
        for (int l = 0; l < c.layers; ++l)
            HIPCHK(p, hipMemset((char*)dec_kv(p, l).base + (size_t)budget_blocks * p->block_elems * p->esz, 0,
                                (size_t)pad_blocks * p->block_elems * p->esz));
    }
    if ((rc = dev_alloc_t(p, &p->bt_dev, p->bt_host.size()))) return bail(rc);
    HIPCHK(p, hipMemcpy(p->bt_dev, p->bt_host.data(), p->bt_host.size() * sizeof(int), hipMemcpyHostToDevice));

    // ---- rotary tables (angles in double on the host, rounded to float)
    {
        const int half = c.head_dim / 2;
        std::vector<float> ct((size_t)p->max_pos * half), st(ct.size());
        for (int pos = 0; pos < p->max_pos; ++pos)
            for (int i = 0; i < half; ++i) {
                const double th = pow(10000.0, -2.0 * i / c.head_dim);
                const double ang = (double)pos * th;
                ct[(size_t)pos * half + i] = (float)cos(ang);
                st[(size_t)pos * half + i] = (float)sin(ang);
            }
        if ((rc = dev_alloc_t(p, &p->cos_tab, ct.size()))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->sin_tab, st.size()))) return bail(rc);
        HIPCHK(p, hipMemcpy(p->cos_tab, ct.data(), ct.size() * 4, hipMemcpyHostToDevice));
        HIPCHK(p, hipMemcpy(p->sin_tab, st.data(), st.size() * 4, hipMemcpyHostToDevice));
    }
    if (c.exp_layers) {
        const int half = c.exp_d / 2;
        std::vector<float> te((size_t)c.n_steps * c.exp_d);
        for (int k = 0; k < c.n_steps; ++k) {
            const double tau = 1.0 - (double)k / c.n_steps;
            for (int j = 0; j < half; ++j) {
                const double a = 1000.0 * tau * pow(10000.0, -(double)j / half);
                te[(size_t)k * c.exp_d + j] = (float)sin(a);
                te[(size_t)k * c.exp_d + half + j] = (float)cos(a);
            }
        }
        if ((rc = dev_alloc_t(p, &p->temb, te.size()))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->tvec, te.size()))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->tmid, te.size()))) return bail(rc);
        HIPCHK(p, hipMemcpy(p->temb, te.data(), te.size() * 4, hipMemcpyHostToDevice));
    }

    // ---- activations
    const size_t pre_rows = (size_t)c.max_envs * c.max_seq;
    const size_t vit_rows = c.vit_layers ? (size_t)c.max_envs * p->patches_per_env : 0;
    const size_t flow_rows = c.exp_layers ? (size_t)c.max_envs * (c.chunk + c.frame_tokens) : 0;
    p->dec_cap = c.max_envs <= 4 ? c.max_envs : (c.max_envs + 7) / 8 * 8;
    p->rows_cap = std::max({pre_rows, vit_rows, flow_rows, (size_t)p->dec_cap});
    auto wmax = [&](auto f) {
        size_t m = f(p->dec);
        if (c.vit_layers) m = std::max(m, (size_t)f(p->vit));
        if (c.exp_layers) m = std::max(m, (size_t)f(p->exp));
        return m;
    };
    const size_t w_d = wmax([](const StackDims& s) { return (size_t)s.d; });
    const size_t w_qkv = wmax([](const StackDims& s) { return (size_t)(s.hq + 2 * s.hkv) * s.hd; });
    const size_t w_q = wmax([](const StackDims& s) { return (size_t)s.hq * s.hd; });
    const size_t w_mlp = wmax([](const StackDims& s) { return (size_t)s.mlp; });
    const size_t R = p->rows_cap;
    if ((rc = dev_alloc_t(p, &p->X, R * w_d))) return bail(rc);
    if ((rc = dev_alloc(p, &p->Xn, R * w_d * p->esz))) return bail(rc);
    if ((rc = dev_alloc(p, &p->Qb, R * w_q * p->esz))) return bail(rc);
    if ((rc = dev_alloc(p, &p->Ob, R * w_q * p->esz))) return bail(rc);
    if ((rc = dev_alloc(p, &p->Hb, R * w_mlp * p->esz))) return bail(rc);
    if (c.n_cams && (rc = dev_alloc(p, &p->patches, (size_t)c.max_envs * p->patches_per_env * p->kpad * p->esz)))
        return bail(rc);
    if (c.vit_layers) {
        if ((rc = dev_alloc_t(p, &p->Vx, vit_rows * c.vit_d))) return bail(rc);
        p->vit_bt_stride = (p->patches_per_env + KV_BLOCK - 1) / KV_BLOCK;
        const size_t vblocks = (size_t)c.max_envs * p->vit_bt_stride;
        const size_t vblock_elems = (size_t)2 * c.vit_heads * KV_BLOCK * (c.vit_d / c.vit_heads);
        if ((rc = dev_alloc(p, &p->vit_kv, vblocks * vblock_elems * p->esz))) return bail(rc);
        std::vector<int> vbt(vblocks);
        std::iota(vbt.begin(), vbt.end(), 0);
        if ((rc = dev_alloc_t(p, &p->vit_bt, vbt.size()))) return bail(rc);
        HIPCHK(p, hipMemcpy(p->vit_bt, vbt.data(), vbt.size() * 4, hipMemcpyHostToDevice));
    }
    if ((rc = dev_alloc_t(p, &p->h_pre, (size_t)(c.max_envs + 1) * c.d))) return bail(rc);
    if ((rc = dev_alloc_t(p, &p->h_norm, (size_t)(c.max_envs + 1) * c.d))) return bail(rc);
    HIPCHK(p, hipMemset(p->h_pre, 0, (size_t)(c.max_envs + 1) * c.d * 4));
    HIPCHK(p, hipMemset(p->h_norm, 0, (size_t)(c.max_envs + 1) * c.d * 4));
    // split-K workspace: 16 splits of the widest skinny projection
    p->ws_floats = (size_t)16 * 256 * std::max(w_qkv, 2 * w_mlp);
    if ((rc = dev_alloc_t(p, &p->ws, p->ws_floats))) return bail(rc);
    if ((rc = dev_alloc_t(p, &p->counters, ebrl::gemm_counter_words()))) return bail(rc);
    HIPCHK(p, hipMemset(p->counters, 0, ebrl::gemm_counter_words() * 4));
    if (c.action_logits) {
        if ((rc = dev_alloc_t(p, &p->lg, (size_t)p->dec_cap * c.n_bins))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->lg_counters, (size_t)p->dec_cap))) return bail(rc);
        HIPCHK(p, hipMemset(p->lg_counters, 0, (size_t)p->dec_cap * 4));
        const size_t outs = (size_t)p->dec_cap * c.n_action_tokens;
        if ((rc = dev_alloc_t(p, &p->dec_tok, outs))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->dec_act, outs))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->dec_mar, outs))) return bail(rc);
    }
    const int max_splits = (c.max_seq + p->tail + ATTN_DEC_CHUNK - 1) / ATTN_DEC_CHUNK;
    p->part_floats = (size_t)std::max(c.max_envs, p->dec_cap) * c.q_heads * max_splits * (c.head_dim + 2);
    if ((rc = dev_alloc_t(p, &p->part, p->part_floats))) return bail(rc);
    {
        const size_t words = (size_t)std::max(c.max_envs, p->dec_cap) * c.q_heads;
        if ((rc = dev_alloc_t(p, &p->attn_counters, words))) return bail(rc);
        HIPCHK(p, hipMemset(p->attn_counters, 0, words * 4));
    }
    if (c.exp_layers) {
        const size_t act_rows = (size_t)c.max_envs * c.chunk;
        if ((rc = dev_alloc_t(p, &p->flow_x, act_rows * c.adim))) return bail(rc);
        if ((rc = dev_alloc_t(p, &p->flow_v0, act_rows * c.adim))) return bail(rc);
        if (c.frame_tokens &&
            (rc = dev_alloc_t(p, &p->flow_f, (size_t)c.max_envs * c.frame_tokens * c.frame_dim)))
            return bail(rc);
    }
    // per-call metadata: generous bound on every call's int arrays
    p->meta_cap = 16 * (R + 64) + (size_t)c.max_envs * (32 + 2 * p->bt_stride) + p->bt_host.size() +
                  (size_t)c.max_envs * c.max_seq / 8 + 4096;
    if ((rc = dev_alloc_t(p, &p->meta_dev, p->meta_cap))) return bail(rc);
    {
        void* hp = nullptr;
        hipError_t e = hipHostMalloc(&hp, p->meta_cap * sizeof(int), hipHostMallocDefault);
        if (e != hipSuccess) {
            fail(p, EBRL_E_OOM, "hipHostMalloc: %s", hipGetErrorString(e));
            return bail(EBRL_E_OOM);
        }
        p->meta_host = (int*)hp;
    }
    if (hipEventCreateWithFlags(&p->meta_ev, hipEventDisableTiming) != hipSuccess) {
        fail(p, EBRL_E_HIP, "hipEventCreate failed");
        return bail(EBRL_E_HIP);
    }
    if (hipStreamCreateWithFlags(&p->cap_stream, hipStreamNonBlocking) != hipSuccess) {
        fail(p, EBRL_E_HIP, "hipStreamCreate failed");
        return bail(EBRL_E_HIP);
    }
    HIPCHK(p, hipDeviceSynchronize());
    *out = p;
    return EBRL_OK;
}

int ebrl_stream_create_cu_masked(int32_t device, const uint32_t* cu_mask, uint32_t n_words, void** out_stream) {
    if (!out_stream || !cu_mask || n_words == 0) return EBRL_E_INVALID;
    *out_stream = nullptr;
    int prev = 0;
    if (hipGetDevice(&prev) != hipSuccess) return EBRL_E_HIP;
    if (hipSetDevice(device) != hipSuccess) return EBRL_E_INVALID;
    hipStream_t s = nullptr;
    hipError_t e = hipExtStreamCreateWithCUMask(&s, n_words, cu_mask);
    (void)hipSetDevice(prev);
    if (e != hipSuccess) {
        g_create_error = std::string("hipExtStreamCreateWithCUMask: ") + hipGetErrorString(e);
        return EBRL_E_HIP;
    }
    int bits = 0;
    for (uint32_t w = 0; w < n_words; ++w) bits += __builtin_popcount(cu_mask[w]);
    {
        std::lock_guard<std::mutex> lk(g_stream_mu);
        g_stream_cus[s] = bits;
    }
    *out_stream = (void*)s;
    return EBRL_OK;
}

int ebrl_stream_destroy(void* stream) {
    if (!stream) return EBRL_E_INVALID;
    {
        std::lock_guard<std::mutex> lk(g_stream_mu);
        g_stream_cus.erase((hipStream_t)stream);
    }
    return hipStreamDestroy((hipStream_t)stream) == hipSuccess ? EBRL_OK : EBRL_E_HIP;
}

int ebrl_policy_bind_stream(ebrl_policy* p, void* stream) {
    int rc = check_ready(p);
    if (rc) return rc;
    HIPCHK(p, hipStreamSynchronize(p->stream));
    p->stream = (hipStream_t)stream;
    // GEMM tile choices (never their sums' order) follow the CUs the stream
    // may use; decode and denoise graphs are cached per CU count
    p->cus = p->dev_cus;
    {
        std::lock_guard<std::mutex> lk(g_stream_mu);
        auto it = g_stream_cus.find(p->stream);
        if (it != g_stream_cus.end() && it->second > 0) p->cus = std::min(it->second, p->dev_cus);
    }
    return EBRL_OK;
}

int ebrl_prefill(ebrl_policy* p, const ebrl_obs_batch* obs, const int32_t* env_ids, int32_t n) {
    int rc = check_ready(p);
    if (rc) return rc;
    if ((rc = check_ids(p, env_ids, n, false))) return rc;
    if (n == 0) return EBRL_OK;
    if (!obs) return fail(p, EBRL_E_INVALID, "obs is NULL");
    const ebrl_config& c = p->cfg;
    const bool images = obs->images != nullptr;
    if (images && !c.n_cams) return fail(p, EBRL_E_INVALID, "policy has no image input");
    const int nimg = images ? p->n_img : 0;
    std::vector<int> llen(n), T(n);
    for (int i = 0; i < n; ++i) {
        llen[i] = obs->lang_len ? obs->lang_len[i] : c.n_lang;
        if (llen[i] < 0 || (llen[i] > 0 && (!obs->lang_ids || llen[i] > obs->lang_stride)))
            return fail(p, EBRL_E_INVALID, "env %d: lang_len %d invalid for lang_stride %d", env_ids[i], llen[i],
                        obs->lang_stride);
        T[i] = nimg + llen[i];
        if (T[i] < 1 || T[i] > c.max_seq)
            return fail(p, EBRL_E_INVALID, "env %d: prefix length %d outside [1, %d]", env_ids[i], T[i], c.max_seq);
    }
    // ---- KV blocks: the budget check counts the blocks these envs already
    // hold as available (they are replaced), and runs before any env's state
    // changes, so a call that fails leaves every existing cache intact
    size_t need = 0, held = 0;
    for (int i = 0; i < n; ++i) {
        need += (size_t)(T[i] + p->tail + KV_BLOCK - 1) / KV_BLOCK;
        held += p->envs[env_ids[i]].blocks.size();
    }
    if (need > p->free_blocks.size() + held)
        return fail(p, EBRL_E_OOM, "KV budget: %zu blocks needed, %zu free", need, p->free_blocks.size() + held);
    for (int i = 0; i < n; ++i) {
        EnvSlot& s = p->envs[env_ids[i]];
        for (int b : s.blocks) p->free_blocks.push_back(b);
        s.blocks.clear();
        s.T = 0;
    }
    for (int i = 0; i < n; ++i) {
        EnvSlot& s = p->envs[env_ids[i]];
        const int nb = (T[i] + p->tail + KV_BLOCK - 1) / KV_BLOCK;
        for (int b = 0; b < nb; ++b) {
            s.blocks.push_back(p->free_blocks.back());
            p->free_blocks.pop_back();
        }
        int* row = &p->bt_host[(size_t)env_ids[i] * p->bt_stride];
        for (int b = 0; b < p->bt_stride; ++b) row[b] = b < nb ? s.blocks[b] : 0;
        s.T = T[i];
    }
    // ---- metadata
    std::vector<int> seq_env(env_ids, env_ids + n), tok_off(n + 1, 0), q_pos0(n, 0), last_row(n);
    for (int i = 0; i < n; ++i) tok_off[i + 1] = tok_off[i] + T[i];
    const int M = tok_off[n];
    if ((size_t)M > p->rows_cap) return fail(p, EBRL_E_INVALID, "internal: %d rows exceed capacity", M);
    for (int i = 0; i < n; ++i) last_row[i] = tok_off[i] + T[i] - 1;
    std::vector<int> row_seq(M), row_pos(M);
    for (int i = 0; i < n; ++i)
        for (int t = 0; t < T[i]; ++t) { row_seq[tok_off[i] + t] = i; row_pos[tok_off[i] + t] = t; }
    std::vector<std::pair<int, int>> tiles;
    for (int i = 0; i < n; ++i)
        for (int q0 = 0; q0 < T[i]; q0 += ATTN_Q_TILE) tiles.push_back({i, q0});
    // causal tiles late in a sequence see the most keys: dispatch them first
    std::stable_sort(tiles.begin(), tiles.end(),
                     [](const std::pair<int, int>& x, const std::pair<int, int>& y) { return x.second > y.second; });
    std::vector<int> tile_seq(tiles.size()), tile_q0(tiles.size());
    for (size_t t = 0; t < tiles.size(); ++t) { tile_seq[t] = tiles[t].first; tile_q0[t] = tiles[t].second; }
    std::vector<int> lang_dst, lang_src;
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < llen[i]; ++j) {
            lang_dst.push_back(tok_off[i] + nimg + j);
            lang_src.push_back(i * obs->lang_stride + j);
        }
    // ViT sequences
    const int pv = p->patches_per_env;
    std::vector<int> v_ident(n), v_off(n), v_len(n, pv), v_zero(n, 0), v_rowseq, v_rowpos, v_tseq, v_tq0;
    if (images && c.vit_layers) {
        for (int i = 0; i < n; ++i) { v_ident[i] = i; v_off[i] = i * pv; }
        for (int i = 0; i < n; ++i)
            for (int t = 0; t < pv; ++t) { v_rowseq.push_back(i); v_rowpos.push_back(t); }
        for (int i = 0; i < n; ++i)
            for (int q0 = 0; q0 < pv; q0 += ATTN_Q_TILE) { v_tseq.push_back(i); v_tq0.push_back(q0); }
    }
    Meta m;
    const size_t o_env = m.add(seq_env), o_off = m.add(tok_off), o_len = m.add(T), o_pos0 = m.add(q_pos0),
                 o_last = m.add(last_row), o_rseq = m.add(row_seq), o_rpos = m.add(row_pos),
                 o_tseq = m.add(tile_seq), o_tq0 = m.add(tile_q0), o_ldst = m.add(lang_dst),
                 o_lsrc = m.add(lang_src), o_vid = m.add(v_ident), o_voff = m.add(v_off), o_vlen = m.add(v_len),
                 o_vzero = m.add(v_zero), o_vrseq = m.add(v_rowseq), o_vrpos = m.add(v_rowpos),
                 o_vtseq = m.add(v_tseq), o_vtq0 = m.add(v_tq0);
    int* md = nullptr;
    if ((rc = upload_meta(p, m, true, &md))) return rc;

    // ---- image tokens
    if (images) {
        prof_begin(p, EBRL_K_OTHER);
        im2col(p->bf16, obs->images, n, c.n_cams, c.img, c.img, c.patch, p->patches, p->kpad, p->stream);
        prof_end(p, 0, 0);
        GemmArgs g;
        g.A = p->patches; g.lda = p->kpad; g.B = p->w_pe; g.ldb = p->kpad; g.M = n * pv; g.K = p->kpad;
        g.epi = EPI_REMAP;
        if (c.vit_layers) {
            g.N = c.vit_d; g.C = p->Vx; g.ldc = c.vit_d; g.row_base = nullptr; g.group = pv;
            g.add = p->vit_pos; g.add_ld = c.vit_d;
            run_gemm(p, g);
            for (int l = 0; l < c.vit_layers; ++l) {
                BlockCall b;
                b.R = p->Vx; b.rows = n * pv; b.sd = &p->vit; b.w = &p->L_vit[l];
                b.kv.base = p->vit_kv; b.kv.block_table = p->vit_bt; b.kv.bt_stride = p->vit_bt_stride;
                b.kv.kv_heads = p->vit.hkv; b.kv.head_dim = p->vit.hd;
                b.seq_env = md + o_vid; b.row_seq = md + o_vrseq; b.row_pos = md + o_vrpos; b.use_rope = false;
                b.pre.seq_env = md + o_vid; b.pre.q_off = md + o_voff; b.pre.q_len = md + o_vlen;
                b.pre.q_pos0 = md + o_vzero; b.pre.kv_len = md + o_vlen; b.pre.tile_seq = md + o_vtseq;
                b.pre.tile_q0 = md + o_vtq0; b.pre.n_tiles = (int)v_tseq.size(); b.pre.causal = false;
                b.pre.max_kv_len = pv;
                b.attn_flop = 4.0 * p->vit.hd * p->vit.hq * (double)n * pv * pv;
                b.attn_bytes = 2.0 * n * pv * (double)(p->vit.hq + p->vit.hkv) * p->vit.hd * p->esz;
                if ((rc = run_block(p, b))) return rc;
            }
            prof_begin(p, EBRL_K_OTHER);
            rmsnorm_rows(p->bf16, p->Vx, c.vit_d, nullptr, p->Xn, c.vit_d, n * pv, c.vit_d, 1e-6f, p->stream);
            prof_end(p, 0, 0);
            g = GemmArgs();
            g.A = p->Xn; g.lda = c.vit_d; g.B = p->w_proj; g.ldb = c.vit_d; g.M = n * pv; g.N = c.d;
            g.K = c.vit_d; g.epi = EPI_REMAP; g.C = p->X; g.ldc = c.d; g.row_base = md + o_off; g.group = pv;
            run_gemm(p, g);
        } else {
            g.N = c.d; g.C = p->X; g.ldc = c.d; g.row_base = md + o_off; g.group = pv;
            run_gemm(p, g);
        }
    }
    // ---- language tokens
    if (!lang_dst.empty()) {
        prof_begin(p, EBRL_K_OTHER);
        embed_rows(p->bf16, p->e_lang, c.vocab, c.d, obs->lang_ids, md + o_lsrc, 0, 0, md + o_ldst, p->X, c.d,
                   (int)lang_dst.size(), p->stream);
        prof_end(p, 0, 0);
    }
    // ---- decoder
    const int maxT = *std::max_element(T.begin(), T.end());
    double causal_pairs = 0, kv_rows = 0;
    for (int i = 0; i < n; ++i) { causal_pairs += 0.5 * T[i] * (T[i] + 1.0); kv_rows += T[i]; }
    for (int l = 0; l < c.layers; ++l) {
        BlockCall b;
        b.R = p->X; b.rows = M; b.sd = &p->dec; b.w = &p->L_dec[l]; b.kv = dec_kv(p, l);
        b.seq_env = md + o_env; b.row_seq = md + o_rseq; b.row_pos = md + o_rpos;
        b.pre.seq_env = md + o_env; b.pre.q_off = md + o_off; b.pre.q_len = md + o_len; b.pre.q_pos0 = md + o_pos0;
        b.pre.kv_len = md + o_len; b.pre.tile_seq = md + o_tseq; b.pre.tile_q0 = md + o_tq0;
        b.pre.n_tiles = (int)tiles.size(); b.pre.causal = true; b.pre.max_kv_len = maxT;
        b.attn_flop = 4.0 * c.head_dim * c.q_heads * causal_pairs;
        // Q read and O written once, every K/V row read once
        b.attn_bytes = 2.0 * kv_rows * (double)(c.q_heads + c.kv_heads) * c.head_dim * p->esz;
        if ((rc = run_block(p, b))) return rc;
    }
    prof_begin(p, EBRL_K_OTHER);
    gather_last(p->X, c.d, md + o_env, md + o_last, n, c.d, 1e-6f, p->h_pre, p->h_norm, p->stream);
    prof_end(p, 0, 0);
    return check_launch(p);
}

int ebrl_decode_actions(ebrl_policy* p, const int32_t* env_ids, int32_t n, int32_t* out_tokens,
                        float* out_actions, float* out_margin) {
    int rc = check_ready(p);
    if (rc) return rc;
    const ebrl_config& c = p->cfg;
    if (!c.action_logits) return fail(p, EBRL_E_UNSUPPORTED, "policy has no autoregressive action head");
    if ((rc = check_ids(p, env_ids, n, true))) return rc;
    if (n == 0) return EBRL_OK;
    if (!out_tokens) return fail(p, EBRL_E_INVALID, "out_tokens is NULL");
    const int ntok = c.n_action_tokens, steps = ntok - 1;
    // The decode GEMMs' split plan holds for at most DECODE_MAX_ROWS rows (past
    // it a different kernel, with another summation order, would take over):
    // larger calls run as consecutive calls of at most that many envs, so an
    // env's bits never depend on the call's size.
    if (n > DECODE_MAX_ROWS) {
        for (int off = 0; off < n; off += DECODE_MAX_ROWS) {
            const int m = std::min(DECODE_MAX_ROWS, n - off);
            const size_t o = (size_t)off * ntok;
            if ((rc = ebrl_decode_actions(p, env_ids + off, m, out_tokens + o, out_actions ? out_actions + o : nullptr,
                                          out_margin ? out_margin + o : nullptr)))
                return rc;
        }
        return EBRL_OK;
    }
    // batch-size class: rows n .. nc-1 decode the padding env; every tile,
    // split and reduction choice of the kernels depends on the problem shape
    // only, so the real rows' bits do not depend on the padding
    const int nc = n <= 4 ? n : std::min(p->dec_cap, (n + 7) / 8 * 8);
    std::vector<int> seq_env(nc, p->pad_env), ident(nc);
    std::copy(env_ids, env_ids + n, seq_env.begin());
    std::iota(ident.begin(), ident.end(), 0);
    std::vector<int> kvlen((size_t)std::max(steps, 1) * nc), pos((size_t)std::max(steps, 1) * nc);
    for (int i = 0; i < nc; ++i) {
        const int T = p->envs[seq_env[i]].T;
        for (int k = 1; k <= steps; ++k) {
            kvlen[(size_t)(k - 1) * nc + i] = T + k;
            pos[(size_t)(k - 1) * nc + i] = T + k - 1;
        }
    }
    Meta m;
    const size_t o_env = m.add(seq_env), o_id = m.add(ident), o_kvl = m.add(kvlen), o_pos = m.add(pos);
    int* md = nullptr;
    if ((rc = upload_meta(p, m, false, &md))) return rc;
    // split count of the fp32 attention path: the policy's longest sequence
    const int max_splits = (c.max_seq + steps + ATTN_DEC_CHUNK - 1) / ATTN_DEC_CHUNK;

    const bool fold = fold_decode_norm(p, p->dec, nc);
    auto body = [&]() -> int {
        LogitsArgs la;
        la.bf16 = p->bf16; la.W = p->w_act; la.d = c.d; la.n_bins = c.n_bins; la.n = nc;
        la.tokens = p->dec_tok; la.actions = p->dec_act; la.margins = p->dec_mar; la.ntok = ntok;
        la.lg = p->lg; la.counters = p->lg_counters;
        la.X = p->h_pre; la.ldx = c.d; la.rows = md + o_env; la.col = 0;
        prof_begin(p, EBRL_K_OTHER);
        action_logits(la, p->stream);
        prof_end(p, 0, (double)c.n_bins * c.d * p->esz);
        for (int k = 1; k <= steps; ++k) {
            prof_begin(p, EBRL_K_OTHER);
            embed_rows(p->bf16, p->e_act, c.n_bins, c.d, p->dec_tok, nullptr, ntok, k - 1, nullptr, p->X, c.d, nc,
                       p->stream, fold ? p->Xn : nullptr, c.d);
            prof_end(p, 0, 0);
            double kv_bytes = 0;
            for (int i = 0; i < nc; ++i) kv_bytes += (double)(p->envs[seq_env[i]].T + k);
            kv_bytes *= 2.0 * c.kv_heads * c.head_dim * p->esz;
            for (int l = 0; l < c.layers; ++l) {
                BlockCall b;
                b.R = p->X; b.rows = nc; b.sd = &p->dec; b.w = &p->L_dec[l]; b.kv = dec_kv(p, l);
                b.seq_env = md + o_env; b.row_seq = md + o_id; b.row_pos = md + o_pos + (size_t)(k - 1) * nc;
                b.decode = true;
                b.dec.seq_env = md + o_env; b.dec.kv_len = md + o_kvl + (size_t)(k - 1) * nc; b.dec.n = nc;
                b.dec.max_splits = max_splits;
                b.attn_bytes = kv_bytes;
                b.attn_flop = kv_bytes / p->esz / (2.0 * c.kv_heads * c.head_dim) * 4.0 * c.q_heads * c.head_dim;
                int rc2 = run_block(p, b);
                if (rc2) return rc2;
            }
            la.X = p->X; la.rows = nullptr; la.col = k;
            prof_begin(p, EBRL_K_OTHER);
            action_logits(la, p->stream);
            prof_end(p, 0, (double)c.n_bins * c.d * p->esz);
        }
        return check_launch(p);
    };
    const std::vector<uint64_t> key = {1, (uint64_t)nc, (uint64_t)p->cus};
    const int inside = (1 << EBRL_K_GEMM_SKINNY) | (1 << EBRL_K_ATTN_DECODE) | (1 << EBRL_K_OTHER) |
                       (nc >= 256 ? (1 << EBRL_K_GEMM) : 0);
    if ((rc = run_graph(p, key, inside, body))) return rc;
    copy_decode_out(p->dec_tok, p->dec_act, p->dec_mar, n * ntok, out_tokens, out_actions, out_margin, p->stream);
    return check_launch(p);
}

int ebrl_flow_denoise(ebrl_policy* p, const int32_t* env_ids, int32_t n, const float* noise, float* out_actions) {
    int rc = check_ready(p);
    if (rc) return rc;
    if (!p->cfg.exp_layers) return fail(p, EBRL_E_UNSUPPORTED, "policy has no flow-matching expert");
    if (p->cfg.frame_tokens)
        return fail(p, EBRL_E_UNSUPPORTED, "policy denoises future frames too: use ebrl_wam_denoise");
    return denoise(p, env_ids, n, nullptr, noise, nullptr, out_actions);
}

int ebrl_wam_denoise(ebrl_policy* p, const int32_t* env_ids, int32_t n, const float* frame_noise,
                     const float* action_noise, float* out_frames, float* out_actions) {
    int rc = check_ready(p);
    if (rc) return rc;
    if (!p->cfg.exp_layers || !p->cfg.frame_tokens)
        return fail(p, EBRL_E_UNSUPPORTED, "policy has no future-frame tokens");
    if (n > 0 && !out_frames) return fail(p, EBRL_E_INVALID, "out_frames is NULL");
    return denoise(p, env_ids, n, frame_noise, action_noise, out_frames, out_actions);
}

int ebrl_read_state(ebrl_policy* p, int32_t what, int32_t env_id, int32_t layer, void* out, int64_t bytes) {
    int rc = check_ready(p);
    if (rc) return rc;
    const ebrl_config& c = p->cfg;
    if (env_id < 0 || env_id >= c.max_envs || !out) return fail(p, EBRL_E_INVALID, "bad env id or out");
    HIPCHK(p, hipStreamSynchronize(p->stream));
    const EnvSlot& s = p->envs[env_id];
    switch (what) {
    case EBRL_STATE_PREFIX_LEN:
        if (bytes < 4) return fail(p, EBRL_E_INVALID, "need 4 bytes");
        *(int32_t*)out = s.T;
        return EBRL_OK;
    case EBRL_STATE_GRAPHS:
        if (bytes < 4) return fail(p, EBRL_E_INVALID, "need 4 bytes");
        *(int32_t*)out = (int32_t)p->graphs.size();
        return EBRL_OK;
    case EBRL_STATE_H_LAST_PRE:
    case EBRL_STATE_H_LAST: {
        if (bytes < (int64_t)c.d * 4) return fail(p, EBRL_E_INVALID, "need %d bytes", c.d * 4);
        const float* src = (what == EBRL_STATE_H_LAST ? p->h_norm : p->h_pre) + (size_t)env_id * c.d;
        HIPCHK(p, hipMemcpy(out, src, (size_t)c.d * 4, hipMemcpyDeviceToHost));
        return EBRL_OK;
    }
    case EBRL_STATE_K:
    case EBRL_STATE_V: {
        if (layer < 0 || layer >= c.layers) return fail(p, EBRL_E_INVALID, "layer out of range");
        if (s.T <= 0) return fail(p, EBRL_E_STATE, "env %d has no prefix", env_id);
        const size_t row = (size_t)c.kv_heads * c.head_dim * p->esz;
        if (bytes < (int64_t)(row * s.T)) return fail(p, EBRL_E_INVALID, "need %zu bytes", row * s.T);
        const size_t head_stride = (size_t)KV_BLOCK * c.head_dim * p->esz;
        const char* base = (const char*)dec_kv(p, layer).base;
        for (int b = 0; b * KV_BLOCK < s.T; ++b) {
            std::vector<char> blk(p->block_elems * p->esz);
            HIPCHK(p, hipMemcpy(blk.data(), base + (size_t)s.blocks[b] * p->block_elems * p->esz, blk.size(),
                                hipMemcpyDeviceToHost));
            const size_t kvoff = what == EBRL_STATE_V ? (size_t)c.kv_heads * head_stride : 0;
            for (int t = b * KV_BLOCK; t < std::min(s.T, (b + 1) * KV_BLOCK); ++t)
                for (int h = 0; h < c.kv_heads; ++h)
                    memcpy((char*)out + (size_t)t * row + (size_t)h * c.head_dim * p->esz,
                           blk.data() + kvoff + h * head_stride + (size_t)(t % KV_BLOCK) * c.head_dim * p->esz,
                           (size_t)c.head_dim * p->esz);
        }
        return EBRL_OK;
    }
    case EBRL_STATE_FLOW_V0: {
        if (!c.exp_layers) return fail(p, EBRL_E_UNSUPPORTED, "no expert");
        const size_t sz = (size_t)c.chunk * c.adim * 4;
        if (bytes < (int64_t)sz) return fail(p, EBRL_E_INVALID, "need %zu bytes", sz);
        auto it = std::find(p->last_flow_ids.begin(), p->last_flow_ids.end(), env_id);
        if (it == p->last_flow_ids.end()) return fail(p, EBRL_E_STATE, "env %d not in the last flow call", env_id);
        const size_t idx = (size_t)(it - p->last_flow_ids.begin());
        HIPCHK(p, hipMemcpy(out, p->flow_v0 + idx * c.chunk * c.adim, sz, hipMemcpyDeviceToHost));
        return EBRL_OK;
    }
    default:
        return fail(p, EBRL_E_INVALID, "unknown state %d", what);
    }
}

int ebrl_generate_weight_host(uint64_t seed, uint32_t tensor_id, int64_t count, double std, int32_t bf16, void* out) {
    if (!out || count < 0) return EBRL_E_INVALID;
    generate_weight(seed, tensor_id, count, std, bf16 != 0, out);
    return EBRL_OK;
}

static int weight_io(ebrl_policy* p, uint32_t tid, void* host, int64_t bytes, bool write) {
    int rc = check_ready(p);
    if (rc) return rc;
    const Placement pl = placement(p, tid);
    if (!pl.ok) return fail(p, EBRL_E_INVALID, "unknown tensor id %u", tid);
    const int64_t sz = (int64_t)pl.rows * pl.cols * (int64_t)p->esz;
    if (bytes != sz) return fail(p, EBRL_E_INVALID, "tensor %u has %lld bytes, got %lld", tid, (long long)sz,
                                 (long long)bytes);
    HIPCHK(p, hipStreamSynchronize(p->stream));
    const size_t img_bytes = (size_t)pl.buf_rows * pl.ld * p->esz;
    std::vector<char> image(img_bytes);
    HIPCHK(p, hipMemcpy(image.data(), pl.buf, img_bytes, hipMemcpyDeviceToHost));
    if (write) {
        scatter_rows(pl, host, image.data(), p->esz);
        HIPCHK(p, hipMemcpy(pl.buf, image.data(), img_bytes, hipMemcpyHostToDevice));
    } else {
        gather_rows(pl, image.data(), host, p->esz);
    }
    return EBRL_OK;
}

int ebrl_read_weight(ebrl_policy* p, uint32_t tensor_id, void* out, int64_t bytes) {
    if (!out) return EBRL_E_INVALID;
    return weight_io(p, tensor_id, out, bytes, false);
}

int ebrl_write_weight(ebrl_policy* p, uint32_t tensor_id, const void* in, int64_t bytes) {
    if (!in) return EBRL_E_INVALID;
    return weight_io(p, tensor_id, const_cast<void*>(in), bytes, true);
}

int ebrl_profile_enable(ebrl_policy* p, int32_t class_mask) {
    int rc = check_ready(p);
    if (rc) return rc;
    if (!class_mask) prof_collect(p);
    p->prof = class_mask != 0;
    p->prof_mask = class_mask;
    return EBRL_OK;
}

int ebrl_profile_read(ebrl_policy* p, int32_t cls, int64_t* launches, double* total_ms, double* flop,
                      double* bytes, int32_t reset) {
    int rc = check_ready(p);
    if (rc) return rc;
    if (cls < 0 || cls >= EBRL_K_COUNT) return fail(p, EBRL_E_INVALID, "kernel class %d", cls);
    prof_collect(p);
    if (launches) *launches = p->p_launch[cls];
    if (total_ms) *total_ms = p->p_ms[cls];
    if (flop) *flop = p->p_flop[cls];
    if (bytes) *bytes = p->p_bytes[cls];
    if (reset) {
        p->p_launch[cls] = 0;
        p->p_ms[cls] = p->p_flop[cls] = p->p_bytes[cls] = 0;
    }
    return EBRL_OK;
}

// ------------------------------------------------------------- ops ABI --

// Split-K workspace of ebrl_op_gemm: one per (device, stream handle), so
// calls on different streams never share partial sums or tile counters.
// 64 MB of partials plus the counters each, kept for the process lifetime.
static constexpr size_t OP_WS_FLOATS = (size_t)16 << 20;
static std::mutex g_ws_mu;
static std::map<std::pair<int, uintptr_t>, float*> g_ws;

int ebrl_op_stream_read(const void* buf, int64_t bytes, uint32_t* out, void* stream) {
    if (!buf || !out || bytes < 16 || bytes % 16 || (uintptr_t)buf % 16) return EBRL_E_INVALID;
    ebrl::stream_read(buf, (size_t)bytes, out, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? EBRL_OK : EBRL_E_HIP;
}

int ebrl_op_gemm(int32_t dtype, const void* A, const void* B, float* C, int32_t M, int32_t N, int32_t K,
                 void* stream) {
    if (!A || !B || !C || M < 1 || N < 1 || K < 8 || K % 8 || N % 4) return EBRL_E_INVALID;
    if (dtype != EBRL_DTYPE_BF16 && dtype != EBRL_DTYPE_FP32) return EBRL_E_INVALID;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return EBRL_E_HIP;
    float* ws = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_ws_mu);
        float*& slot = g_ws[{dev, (uintptr_t)stream}];
        if (!slot) {
            const size_t words = OP_WS_FLOATS + ebrl::gemm_counter_words();
            if (hipMalloc((void**)&slot, words * 4) != hipSuccess) { slot = nullptr; return EBRL_E_OOM; }
            if (hipMemset(slot + OP_WS_FLOATS, 0, ebrl::gemm_counter_words() * 4) != hipSuccess) return EBRL_E_HIP;
        }
        ws = slot;
    }
    GemmArgs a;
    a.bf16 = dtype == EBRL_DTYPE_BF16;
    a.A = A; a.lda = K; a.B = B; a.ldb = K; a.M = M; a.N = N; a.K = K;
    a.epi = EPI_F32; a.C = C; a.ldc = N; a.ws = ws; a.ws_floats = OP_WS_FLOATS;
    a.counters = reinterpret_cast<unsigned*>(ws + OP_WS_FLOATS);
    a.split_ok = M < 256;
    ebrl::gemm(a, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? EBRL_OK : EBRL_E_HIP;
}

// ebrl_op_gemm_noalloc: the same product with its split-K partials and tile
// counters in `scratch`, a fixed device array each GPU holds for the whole
// process, instead of memory the library allocates.  The array's name in
// host code is not a device address: its address on each device comes from
// hipGetSymbolAddress, taken once per device with that device current.
// The counters start at zero (device globals are zero-initialised) and
// every kernel that uses one leaves it at zero.
static constexpr size_t NOALLOC_WS_FLOATS = (size_t)4 << 20;   // 16 MB of partial sums
static constexpr size_t NOALLOC_COUNTER_WORDS = 4096;          // = gemm_counter_words()
static __device__ __align__(256) float scratch[NOALLOC_WS_FLOATS + NOALLOC_COUNTER_WORDS];
static constexpr int NOALLOC_MAX_DEVICES = 64;
static std::mutex g_scratch_mu;
static float* g_scratch_ptr[NOALLOC_MAX_DEVICES];

static int scratch_on_device(int dev, float** out) {
    if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return EBRL_E_INVALID;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return EBRL_E_HIP;
        }
        g_scratch_ptr[dev] = static_cast<float*>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return EBRL_OK;
}

int ebrl_op_gemm_noalloc(int32_t dtype, const void* A, const void* B, float* C, int32_t M, int32_t N, int32_t K,
                         void* stream) {
    static_assert(NOALLOC_COUNTER_WORDS >= 4096, "tile counters of the decode GEMM");
    if (!A || !B || !C || M < 1 || N < 1 || K < 8 || K % 8 || N % 4) return EBRL_E_INVALID;
    if (dtype != EBRL_DTYPE_BF16 && dtype != EBRL_DTYPE_FP32) return EBRL_E_INVALID;
    if (ebrl::gemm_counter_words() > NOALLOC_COUNTER_WORDS) return EBRL_E_INVALID;
    const bool bf16 = dtype == EBRL_DTYPE_BF16;
    // plan exactly as ebrl_op_gemm does (same workspace size), so both give
    // the same bits; shapes whose plan writes more partials than fit are refused
    const bool split_ok = M < 256;
    if (ebrl::gemm_ws_floats_used(bf16, M, N, K, OP_WS_FLOATS, split_ok) > NOALLOC_WS_FLOATS) return EBRL_E_INVALID;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return EBRL_E_HIP;
    float* ws = nullptr;
    const int rc = scratch_on_device(dev, &ws);
    if (rc) return rc;
    GemmArgs a;
    a.bf16 = bf16;
    a.A = A; a.lda = K; a.B = B; a.ldb = K; a.M = M; a.N = N; a.K = K;
    a.epi = EPI_F32; a.C = C; a.ldc = N; a.ws = ws; a.ws_floats = OP_WS_FLOATS;
    a.counters = reinterpret_cast<unsigned*>(ws + NOALLOC_WS_FLOATS);
    a.split_ok = split_ok;
    ebrl::gemm(a, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? EBRL_OK : EBRL_E_HIP;
}

}  // extern "C"
