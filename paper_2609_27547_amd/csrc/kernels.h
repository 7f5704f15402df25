// Launch wrappers of the GPU library's kernels (host-callable).
#pragma once

#include <algorithm>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace ebrl {

// ------------------------------------------------------------------ GEMM --
enum EpiKind {
    EPI_F32 = 0,     // C f32 [M, ldc] = acc
    EPI_ACT = 1,     // C act dtype = acc (bf16 or f32)
    EPI_RESID = 2,   // C f32 += acc (residual stream)
    EPI_REMAP = 3,   // C f32 row row_base[m/group] + m%group = acc (+ add row m%group)
    EPI_SWIGLU = 4,  // packed gate/up -> C act [M, N/2] = silu(gate) * up
    EPI_QKV = 5      // rotary-paired Q/K/V rows -> rotated Q (act) + paged K/V cache (see RopeKVArgs)
};
struct RopeKVArgs;

struct GemmArgs {
    bool bf16 = true;
    const void* A = nullptr; int lda = 0;   // [M, K] activations
    const void* B = nullptr; int ldb = 0;   // [N, K] weights
    int M = 0, N = 0, K = 0;
    EpiKind epi = EPI_F32;
    void* C = nullptr; int ldc = 0;
    const int* row_base = nullptr; int group = 1;
    const void* add = nullptr; int add_ld = 0;
    const RopeKVArgs* rope = nullptr;           // EPI_QKV parameters
    float* ws = nullptr; size_t ws_floats = 0;  // split-K workspace
    // gemm_counter_words() zeroed words; bf16 GEMMs with K splits leave them
    // zero again.  Calls that share a workspace must not overlap in time.
    unsigned* counters = nullptr;
    // Decode GEMMs (M = batch, at most 256) may split K; the split count then
    // depends on (N, K) only, so an element's summation order -- and its bits
    // -- do not depend on the batch size.  Without splitting, every kernel
    // variant sums K in the same 64-wide steps, so results do not depend on M
    // either.
    bool split_ok = false;
    // Decode GEMMs with a paired epilogue (EPI_QKV, EPI_SWIGLU) and one K
    // split (gemm_row_norm_ok): A holds un-normalised rows in bf16 and every
    // output row is scaled by 1/sqrt(mean_k A[m][k]^2 + norm_eps), i.e. the
    // unit-gain RMSNorm of the input folded into the projection.
    bool row_norm = false; float norm_eps = 1e-6f;
    // EPI_RESID: also store the updated rows in bf16 here (nullable).
    void* xb = nullptr; int ldxb = 0;
    // Compute units the launch stream may use (its CU mask): the decode
    // kernel's column-slice width and the large-M kernel's macro tile are
    // priced in rounds over this many CUs.  Neither choice changes an
    // element's summation order.
    int cus = 256;
};
// Decode GEMMs (split_ok) plan their K splits for at most this many rows;
// callers that need batch-size-independent bits keep calls within it.
constexpr int DECODE_MAX_ROWS = 256;
// Returns the number of K splits used (1 = single pass).
int gemm(const GemmArgs& a, hipStream_t s);
int gemm_splits(bool bf16, int M, int N, int K, size_t ws_floats, bool split_ok);
bool gemm_row_norm_ok(bool bf16, int M, int N, int K, size_t ws_floats);
size_t gemm_counter_words();
// Workspace floats the plan for (M, N, K) writes (0 without a K split).
size_t gemm_ws_floats_used(bool bf16, int M, int N, int K, size_t ws_floats, bool split_ok);

// ------------------------------------------------------------- attention --
// Paged KV: layer base pointer; physical block b holds
// [2 (K, V)][kv_heads][16 tokens][head_dim] elements.
struct PagedKV {
    void* base = nullptr;            // this layer's first block
    const int* block_table = nullptr;  // [max_envs][bt_stride]
    int bt_stride = 0;
    int kv_heads = 0, head_dim = 0;
};

// Flash attention over query tiles of ATTN_Q_TILE rows.  Tile t covers rows
// [tile_q0[t], +ATTN_Q_TILE) of sequence tile_seq[t].
constexpr int ATTN_Q_TILE = 64;
struct AttnPrefillArgs {
    bool bf16 = true;
    const void* Q = nullptr; int ldq = 0;  // [rows, q_heads*hd]
    void* O = nullptr; int ldo = 0;        // [rows, q_heads*hd]
    int q_heads = 0;
    PagedKV kv;
    const int* seq_env = nullptr;   // [n] block-table row of each sequence
    const int* q_off = nullptr;     // [n] first Q/O row
    const int* q_len = nullptr;     // [n]
    const int* q_pos0 = nullptr;    // [n] absolute position of the first query
    const int* kv_len = nullptr;    // [n]
    const int* tile_seq = nullptr;  // [n_tiles]
    const int* tile_q0 = nullptr;   // [n_tiles]
    int n_tiles = 0;
    bool causal = true;
    int max_kv_len = 0;             // fp32 path: scores buffer size
};
void attn_prefill(const AttnPrefillArgs& a, hipStream_t s);
// bf16 attention kernels stage a sequence's block table in LDS: at most this
// many 16-token blocks (4096 tokens) per sequence.
constexpr int ATTN_BT_MAX = 256;

// One query per sequence against kv_len[i] keys, split over the sequence in
// chunks (fp32: ATTN_DEC_CHUNK keys; bf16: at most 512 keys at head dim 128,
// 1024 at 64) merged in chunk order.
constexpr int ATTN_DEC_CHUNK = 64;
struct AttnDecodeArgs {
    bool bf16 = true;
    const void* Q = nullptr; int ldq = 0;  // [n, q_heads*hd]
    void* O = nullptr; int ldo = 0;
    int q_heads = 0;
    PagedKV kv;
    const int* seq_env = nullptr;
    const int* kv_len = nullptr;
    int n = 0;
    int max_splits = 0;            // ceil(longest kv_len / ATTN_DEC_CHUNK) the buffers are sized for
    float* part = nullptr;         // [n][q_heads][max_splits][hd + 2]
    // bf16: [n][q_heads] zeroed words (left zero after the call)
    unsigned* counters = nullptr;
};
void attn_decode(const AttnDecodeArgs& a, hipStream_t s);

// ----------------------------------------------------------------- misc --
// Y[row] = rmsnorm(X[src_row]) ; src_row = rows ? rows[i] : i
void rmsnorm_rows(bool bf16_out, const float* X, int ldx, const int* rows, void* Y, int ldy,
                  int n_rows, int d, float eps, hipStream_t s);

// Rotary embedding + paged KV write of the fused QKV projection, applied in
// the GEMM epilogue (EPI_QKV): rotated queries go to Q (act dtype), rotated
// keys and the values to the paged cache at (seq_env[row_seq[m]],
// row_pos[m]).  use_rope = false skips rotation.  The QKV weight rows are
// packed per head so that rows e and e + hd/2 sit in the two 16-row halves
// of one 32-row group.  (qkv/ld are used only by the standalone kernel.)
struct RopeKVArgs {
    bool bf16 = true;
    const float* qkv = nullptr; int ld = 0;
    int M = 0, q_heads = 0;
    void* Q = nullptr; int ldq = 0;
    PagedKV kv;
    const int* seq_env = nullptr;
    const int* row_seq = nullptr;
    const int* row_pos = nullptr;
    const float* cos_tab = nullptr;  // [max_pos][hd/2]
    const float* sin_tab = nullptr;
    bool use_rope = true;
};
void rope_kv_write(const RopeKVArgs& a, hipStream_t s);

// X[dst] = E[id] as float (id = ids[src ? src[i] : i*stride + off]; dst = dst_rows ? dst_rows[i] : i);
// ids outside [0, n_rows_e) give zero rows.
// xb (nullable, bf16 policies): the same rows in bf16 as well.
void embed_rows(bool bf16, const void* E, int n_rows_e, int d, const int* ids, const int* src, int stride,
                int off, const int* dst_rows, float* X, int ldx, int n, hipStream_t s, void* xb = nullptr,
                int ldxb = 0);

// images f32 [n, cams, H, W, 3] -> patches [n*cams*(H/P)*(W/P), kpad] (zero-padded columns)
void im2col(bool bf16, const float* img, int n, int cams, int H, int W, int P, void* out,
            int kpad, hipStream_t s);

// Action head: logits = W_act . rmsnorm(x_row), argmax (ties -> lowest), top-2 margin,
// bin -> action.  Writes column `col` of [n, ntok] outputs.
struct LogitsArgs {
    bool bf16 = true;
    const float* X = nullptr; int ldx = 0;
    const int* rows = nullptr;      // gather rows of X (nullable: identity)
    const void* W = nullptr;        // [n_bins, d]
    int d = 0, n_bins = 256, n = 0;
    float eps = 1e-6f;
    int* tokens = nullptr; float* actions = nullptr; float* margins = nullptr;
    int ntok = 7, col = 0;
    // bf16 heads with d % 512 == 0 and n_bins % 64 == 0: logits scratch
    // [n][n_bins] and n zeroed per-row counters (left zero after the call)
    float* lg = nullptr; unsigned* counters = nullptr;
};
void action_logits(const LogitsArgs& a, hipStream_t s);

// Streaming read of `bytes` (multiple of 16) with non-temporal loads (HBM read reference).
void stream_read(const void* buf, size_t bytes, unsigned* out, hipStream_t s);

// Last prefix row of each sequence: h_pre[env] = X[row]; h_norm[env] = rmsnorm(X[row]).
void gather_last(const float* X, int ldx, const int* seq_env, const int* last_row, int n, int d,
                 float eps, float* h_pre, float* h_norm, hipStream_t s);

// out[r][n] = sum_k in[r][k] * W[n][k]  (W act dtype), optional silu on the input.
void small_linear(bool bf16, const float* in, int R, int K, const void* W, int N, float* out,
                  bool silu_input, hipStream_t s);

// Flow-matching input projection (+ time vector) and output head + Euler
// update of one denoised modality; its token r lives in row
// (r / per_in) * per_out + off + r % per_in of H.
void flow_in(bool bf16, const float* x, int rows, int adim, const void* W_ain, const float* tvec,
             int d, float* H, int ldh, int per_in, int per_out, int off, hipStream_t s);
void flow_out(bool bf16, const float* H, int ldh, int rows, int d, const void* W_aout, int adim,
              float eps, float n_steps, float* x, float* v_out, int per_in, int per_out, int off,
              hipStream_t s);

// Element copy (device) with f32 -> f32.
void copy_f32(const float* src, float* dst, size_t n, hipStream_t s);
// The first `count` elements of a decode call's tokens (and, where the
// destination is not NULL, actions and margins) to the caller's buffers.
void copy_decode_out(const int* tok, const float* act, const float* mar, int count, int* out_tok, float* out_act,
                     float* out_mar, hipStream_t s);
// Standard normals for `rows` rows of per_row floats: Philox4x32-10 with
// counter (pair, calls[i], env[i], stream) under the seed, Box-Muller.
void normal_noise(float* out, int rows, int per_row, const int* env, const int* calls, uint64_t seed,
                  uint32_t stream, hipStream_t s);

}  // namespace ebrl
