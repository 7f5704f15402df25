// Row-wise kernels of the policy forward: RMSNorm, rotary embedding with the
// paged-KV write, embedding gathers, patch extraction, the 256-bin action
// head with its argmax, and the flow-matching expert's input and Euler
// update.  All reductions run in a fixed order (deterministic results).
#include <math.h>

#include <type_traits>

#include "kernels.h"

namespace ebrl {

template <typename T> EBRL_DEV void load8v(const T* p, float* o);
template <> EBRL_DEV void load8v<bf16_t>(const bf16_t* p, float* o) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        o[2 * i] = __uint_as_float(w[i] << 16);
        o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}
template <> EBRL_DEV void load8v<float>(const float* p, float* o) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}

// sum of squares of a row (fixed order), then 1/sqrt(mean + eps)
EBRL_DEV float row_rstd(const float* x, int d, float eps, float* red) {
    float ss = 0.f;
    for (int j = threadIdx.x * 4; j < d; j += blockDim.x * 4) {
        const float4 v = *reinterpret_cast<const float4*>(x + j);
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    ss = block_sum(ss, red);
    return 1.0f / sqrtf(ss / (float)d + eps);
}

// ------------------------------------------------------------- RMSNorm --
template <typename TO>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* X, int ldx, const int* rows, TO* Y,
                                                      int ldy, int d, float eps)
{
    __shared__ float red[16];
    const int i = blockIdx.x;
    const int src = rows ? rows[i] : i;
    const float* x = X + (size_t)src * ldx;
    const float rs = row_rstd(x, d, eps, red);
    TO* y = Y + (size_t)i * ldy;
    for (int j = threadIdx.x * 4; j < d; j += blockDim.x * 4) {
        const float4 v = *reinterpret_cast<const float4*>(x + j);
        st4<TO>(y + j, v.x * rs, v.y * rs, v.z * rs, v.w * rs);
    }
}

// One wave per row for d % 256 == 0: the row stays in registers (NV float4
// per lane, lane-interleaved so each load instruction reads 1 KB of the row),
// the sum of squares is a wave reduction, no workgroup barrier.
template <typename TO, int NV>
__global__ __launch_bounds__(256) void rmsnorm_wave_kernel(const float* X, int ldx, const int* rows, TO* Y,
                                                           int ldy, int n_rows, int d, float eps)
{
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int src = rows ? rows[i] : i;
    const float* x = X + (size_t)src * ldx;
    float4 v[NV];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        v[k] = *reinterpret_cast<const float4*>(x + (k * 64 + lane) * 4);
        ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
    }
    ss = wave_sum(ss);
    const float rs = 1.0f / sqrtf(ss / (float)d + eps);
    TO* y = Y + (size_t)i * ldy;
#pragma unroll
    for (int k = 0; k < NV; ++k)
        st4<TO>(y + (k * 64 + lane) * 4, v[k].x * rs, v[k].y * rs, v[k].z * rs, v[k].w * rs);
}

template <typename TO>
static bool rmsnorm_wave(const float* X, int ldx, const int* rows, TO* Y, int ldy, int n_rows, int d,
                         float eps, hipStream_t s) {
    if (d % 256) return false;
    const dim3 grid((n_rows + 3) / 4), block(256);
    switch (d / 256) {
    case 1: hipLaunchKernelGGL((rmsnorm_wave_kernel<TO, 1>), grid, block, 0, s, X, ldx, rows, Y, ldy, n_rows, d, eps); return true;
    case 2: hipLaunchKernelGGL((rmsnorm_wave_kernel<TO, 2>), grid, block, 0, s, X, ldx, rows, Y, ldy, n_rows, d, eps); return true;
    case 4: hipLaunchKernelGGL((rmsnorm_wave_kernel<TO, 4>), grid, block, 0, s, X, ldx, rows, Y, ldy, n_rows, d, eps); return true;
    case 8: hipLaunchKernelGGL((rmsnorm_wave_kernel<TO, 8>), grid, block, 0, s, X, ldx, rows, Y, ldy, n_rows, d, eps); return true;
    case 16: hipLaunchKernelGGL((rmsnorm_wave_kernel<TO, 16>), grid, block, 0, s, X, ldx, rows, Y, ldy, n_rows, d, eps); return true;
    default: return false;
    }
}

void rmsnorm_rows(bool bf16_out, const float* X, int ldx, const int* rows, void* Y, int ldy,
                  int n_rows, int d, float eps, hipStream_t s) {
    if (n_rows <= 0) return;
    if (bf16_out ? rmsnorm_wave<bf16_t>(X, ldx, rows, (bf16_t*)Y, ldy, n_rows, d, eps, s)
                 : rmsnorm_wave<float>(X, ldx, rows, (float*)Y, ldy, n_rows, d, eps, s))
        return;
    if (bf16_out)
        hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(n_rows), dim3(256), 0, s, X, ldx, rows,
                           (bf16_t*)Y, ldy, d, eps);
    else
        hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(n_rows), dim3(256), 0, s, X, ldx, rows,
                           (float*)Y, ldy, d, eps);
}

// ------------------------------------------------------ rotary + KV write --
template <typename T>
__global__ __launch_bounds__(256) void rope_kv_kernel(RopeKVArgs a)
{
    const int m = blockIdx.x;
    const int hd = a.kv.head_dim, half = hd / 2;
    const int hq = a.q_heads, hkv = a.kv.kv_heads;
    const int seq = a.row_seq[m], pos = a.row_pos[m];
    const int env = a.seq_env[seq];
    const float* x = a.qkv + (size_t)m * a.ld;
    const float* ct = a.cos_tab + (size_t)pos * half;
    const float* st = a.sin_tab + (size_t)pos * half;
    const int blk = a.kv.block_table[(size_t)env * a.kv.bt_stride + (pos >> 4)];
    T* kdst = (T*)a.kv.base + (size_t)blk * 2 * hkv * KV_BLOCK * hd + (size_t)(pos & 15) * hd;
    T* vdst = kdst + (size_t)hkv * KV_BLOCK * hd;
    T* q = (T*)a.Q + (size_t)m * a.ldq;
    // rotated queries
    for (int idx = threadIdx.x; idx < hq * half; idx += blockDim.x) {
        const int h = idx / half, i = idx - h * half;
        const float x1 = x[h * hd + i], x2 = x[h * hd + i + half];
        float o1 = x1, o2 = x2;
        if (a.use_rope) {
            const float c = ct[i], sn = st[i];
            o1 = x1 * c - x2 * sn;
            o2 = x2 * c + x1 * sn;
        }
        st_elem<T>(q + h * hd + i, o1);
        st_elem<T>(q + h * hd + i + half, o2);
    }
    // rotated keys
    const float* xk = x + hq * hd;
    for (int idx = threadIdx.x; idx < hkv * half; idx += blockDim.x) {
        const int h = idx / half, i = idx - h * half;
        const float x1 = xk[h * hd + i], x2 = xk[h * hd + i + half];
        float o1 = x1, o2 = x2;
        if (a.use_rope) {
            const float c = ct[i], sn = st[i];
            o1 = x1 * c - x2 * sn;
            o2 = x2 * c + x1 * sn;
        }
        T* kd = kdst + (size_t)h * KV_BLOCK * hd;
        st_elem<T>(kd + i, o1);
        st_elem<T>(kd + i + half, o2);
    }
    // values
    const float* xv = x + (hq + hkv) * hd;
    for (int idx = threadIdx.x; idx < hkv * hd; idx += blockDim.x) {
        const int h = idx / hd, i = idx - h * hd;
        st_elem<T>(vdst + (size_t)h * KV_BLOCK * hd + i, xv[idx]);
    }
}

void rope_kv_write(const RopeKVArgs& a, hipStream_t s) {
    if (a.M <= 0) return;
    if (a.bf16) hipLaunchKernelGGL(rope_kv_kernel<bf16_t>, dim3(a.M), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(rope_kv_kernel<float>, dim3(a.M), dim3(256), 0, s, a);
}

// ------------------------------------------------------------ embedding --
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const T* E, int n_rows_e, int d, const int* ids,
                                                    const int* src, int stride, int off, const int* dst_rows,
                                                    float* X, int ldx, bf16_t* xb, int ldxb)
{
    const int i = blockIdx.x;
    const int id = ids[src ? src[i] : i * stride + off];
    const int dst = dst_rows ? dst_rows[i] : i;
    float* x = X + (size_t)dst * ldx;
    bf16_t* y = xb ? xb + (size_t)dst * ldxb : nullptr;
    if (id < 0 || id >= n_rows_e) {  // out-of-range ids embed as zero rows
        for (int j = threadIdx.x; j < d; j += blockDim.x) {
            x[j] = 0.f;
            if (y) y[j] = 0;
        }
        return;
    }
    const T* e = E + (size_t)id * d;
    for (int j = threadIdx.x; j < d; j += blockDim.x) {
        const float v = ld_elem<T>(e + j);
        x[j] = v;
        if (y) st_elem<bf16_t>(y + j, v);
    }
}

void embed_rows(bool bf16, const void* E, int n_rows_e, int d, const int* ids, const int* src, int stride,
                int off, const int* dst_rows, float* X, int ldx, int n, hipStream_t s, void* xb, int ldxb) {
    if (n <= 0) return;
    if (bf16)
        hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(n), dim3(256), 0, s, (const bf16_t*)E, n_rows_e, d,
                           ids, src, stride, off, dst_rows, X, ldx, (bf16_t*)xb, ldxb);
    else
        hipLaunchKernelGGL(embed_kernel<float>, dim3(n), dim3(256), 0, s, (const float*)E, n_rows_e, d,
                           ids, src, stride, off, dst_rows, X, ldx, (bf16_t*)nullptr, 0);
}

// ----------------------------------------------------------- patchify --
// One thread per 8 consecutive K elements of a patch row (a 16-byte bf16
// store); 32-bit index arithmetic.  kpad % 8 == 0; K elements past P*P*3 are
// the zero padding.
template <typename T>
__global__ __launch_bounds__(256) void im2col_kernel(const float* img, int rows, int cams, int H, int W, int P,
                                                     T* out, int kpad)
{
    const int gw = W / P, np = (H / P) * gw;
    const int kreal = P * P * 3, kc = kpad / 8;
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= rows * kc) return;
    const int row = e / kc, k0 = (e - row * kc) * 8;
    const int env = row / (cams * np), p = row - env * cams * np;
    const int cam = p / np, pp = p - cam * np;
    const int py = pp / gw, px = pp - py * gw;
    const float* base = img + ((size_t)(env * cams + cam) * H + py * P) * W * 3 + (size_t)px * P * 3;
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int k = k0 + j;
        v[j] = 0.f;
        if (k < kreal) {
            const int dy = k / (3 * P), rem = k - dy * 3 * P;
            v[j] = base[(size_t)dy * W * 3 + rem];
        }
    }
    st4<T>(out + (size_t)e * 8, v[0], v[1], v[2], v[3]);
    st4<T>(out + (size_t)e * 8 + 4, v[4], v[5], v[6], v[7]);
}

void im2col(bool bf16, const float* img, int n, int cams, int H, int W, int P, void* out, int kpad,
            hipStream_t s) {
    const long rows = (long)n * cams * (H / P) * (W / P);
    if (rows <= 0) return;
    const long threads = rows * (kpad / 8);
    const int blocks = (int)((threads + 255) / 256);
    if (bf16)
        hipLaunchKernelGGL(im2col_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, img, (int)rows, cams, H, W, P,
                           (bf16_t*)out, kpad);
    else
        hipLaunchKernelGGL(im2col_kernel<float>, dim3(blocks), dim3(256), 0, s, img, (int)rows, cams, H, W, P,
                           (float*)out, kpad);
}

// --------------------------------------------------------- action head --
template <typename TW>
__global__ __launch_bounds__(256) void logits_kernel(LogitsArgs a)
{
    extern __shared__ float sh[];
    float* hn = sh;              // [d]
    float* lg = sh + a.d;        // [n_bins]
    __shared__ float red[16];
    const int i = blockIdx.x;
    const int src = a.rows ? a.rows[i] : i;
    const float* x = a.X + (size_t)src * a.ldx;
    const float rs = row_rstd(x, a.d, a.eps, red);
    for (int j = threadIdx.x; j < a.d; j += blockDim.x) hn[j] = x[j] * rs;
    __syncthreads();
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
    const TW* W = (const TW*)a.W;
    for (int b = wave; b < a.n_bins; b += nw) {
        float dot = 0.f;
        for (int j = lane * 8; j < a.d; j += 512) {
            float w[8];
            load8v<TW>(W + (size_t)b * a.d + j, w);
#pragma unroll
            for (int u = 0; u < 8; ++u) dot = fmaf(w[u], hn[j + u], dot);
        }
        dot = wave_sum(dot);
        if (lane == 0) lg[b] = dot;
    }
    __syncthreads();
    if (wave == 0) {
        // argmax, ties to the lowest index
        float bv = -INFINITY;
        int bi = 0x7fffffff;
        for (int b = lane; b < a.n_bins; b += 64) {
            const float v = lg[b];
            if (v > bv || (v == bv && b < bi)) { bv = v; bi = b; }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const float ov = __shfl_xor(bv, off, 64);
            const int oi = __shfl_xor(bi, off, 64);
            if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
        }
        float sv = -INFINITY;
        for (int b = lane; b < a.n_bins; b += 64)
            if (b != bi) sv = fmaxf(sv, lg[b]);
        sv = wave_max(sv);
        if (lane == 0) {
            const int o = i * a.ntok + a.col;
            a.tokens[o] = bi;
            if (a.actions) a.actions[o] = -1.0f + (2.0f * (float)bi + 1.0f) / (float)a.n_bins;
            if (a.margins) a.margins[o] = bv - sv;
        }
    }
}

// bf16 action head, split over bins: grid (row, n_bins / 64).  A workgroup
// normalises its row (RMSNorm, gains 1) into LDS, each wave takes 16 bins and
// loads their weight rows in one burst per 512 columns; the row's logits go
// to a scratch row, and the last of the row's workgroups (device-scope
// counter) takes the argmax (ties to the lowest bin) and the top-2 margin.
__global__ __launch_bounds__(256) void logits_split_kernel(LogitsArgs a)
{
    extern __shared__ float hn[];   // [d]
    __shared__ float red[16];
    __shared__ int s_last;
    const int i = blockIdx.x, part = blockIdx.y;
    const int src = a.rows ? a.rows[i] : i;
    const float* x = a.X + (size_t)src * a.ldx;
    const float rs = row_rstd(x, a.d, a.eps, red);
    for (int j = threadIdx.x; j < a.d; j += blockDim.x) hn[j] = x[j] * rs;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int b0 = part * 64 + wave * 16;
    const bf16_t* W = (const bf16_t*)a.W + (size_t)b0 * a.d + lane * 8;
    float acc[16];
#pragma unroll
    for (int b = 0; b < 16; ++b) acc[b] = 0.f;
    for (int c = 0; c < a.d; c += 512) {
        uint4 w[16];
#pragma unroll
        for (int b = 0; b < 16; ++b) w[b] = *reinterpret_cast<const uint4*>(W + (size_t)b * a.d + c);
        float h[8];
        const float4 h0 = *reinterpret_cast<const float4*>(hn + c + lane * 8);
        const float4 h1 = *reinterpret_cast<const float4*>(hn + c + lane * 8 + 4);
        h[0] = h0.x; h[1] = h0.y; h[2] = h0.z; h[3] = h0.w; h[4] = h1.x; h[5] = h1.y; h[6] = h1.z; h[7] = h1.w;
#pragma unroll
        for (int b = 0; b < 16; ++b) {
            float wf[8];
            load8v<bf16_t>(reinterpret_cast<const bf16_t*>(&w[b]), wf);
#pragma unroll
            for (int u = 0; u < 8; ++u) acc[b] = fmaf(wf[u], h[u], acc[b]);
        }
    }
    const __amdgpu_buffer_rsrc_t lgr = coherent_rsrc(a.lg + (size_t)i * a.n_bins);
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        const float v = wave_sum(acc[b]);
        if (lane == b) st_coherent1(lgr, (b0 + b) * 4, v);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0)
        s_last = __hip_atomic_fetch_add(a.counters + i, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                 (unsigned)(gridDim.y - 1);
    __syncthreads();
    if (!s_last || wave != 0) return;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int b = lane; b < a.n_bins; b += 64) {
        const float v = ld_coherent1(lgr, b * 4);
        if (v > bv || (v == bv && b < bi)) { bv = v; bi = b; }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bv, off, 64);
        const int oi = __shfl_xor(bi, off, 64);
        if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    float sv = -INFINITY;
    for (int b = lane; b < a.n_bins; b += 64)
        if (b != bi) sv = fmaxf(sv, ld_coherent1(lgr, b * 4));
    sv = wave_max(sv);
    if (lane == 0) {
        const int o = i * a.ntok + a.col;
        a.tokens[o] = bi;
        if (a.actions) a.actions[o] = -1.0f + (2.0f * (float)bi + 1.0f) / (float)a.n_bins;
        if (a.margins) a.margins[o] = bv - sv;
        __hip_atomic_store(a.counters + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

void action_logits(const LogitsArgs& a, hipStream_t s) {
    if (a.n <= 0) return;
    if (a.bf16 && a.lg && a.counters && a.d % 512 == 0 && a.n_bins % 64 == 0) {
        hipLaunchKernelGGL(logits_split_kernel, dim3(a.n, a.n_bins / 64), dim3(256),
                           (size_t)a.d * sizeof(float), s, a);
        return;
    }
    const size_t shm = (size_t)(a.d + a.n_bins) * sizeof(float);
    if (a.bf16) hipLaunchKernelGGL(logits_kernel<bf16_t>, dim3(a.n), dim3(256), shm, s, a);
    else hipLaunchKernelGGL(logits_kernel<float>, dim3(a.n), dim3(256), shm, s, a);
}

// ---------------------------------------------------- last prefix row --
__global__ __launch_bounds__(256) void gather_last_kernel(const float* X, int ldx, const int* seq_env,
                                                          const int* last_row, int d, float eps,
                                                          float* h_pre, float* h_norm)
{
    __shared__ float red[16];
    const int i = blockIdx.x;
    const float* x = X + (size_t)last_row[i] * ldx;
    const int env = seq_env[i];
    const float rs = row_rstd(x, d, eps, red);
    for (int j = threadIdx.x; j < d; j += blockDim.x) {
        h_pre[(size_t)env * d + j] = x[j];
        h_norm[(size_t)env * d + j] = x[j] * rs;
    }
}

void gather_last(const float* X, int ldx, const int* seq_env, const int* last_row, int n, int d,
                 float eps, float* h_pre, float* h_norm, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(gather_last_kernel, dim3(n), dim3(256), 0, s, X, ldx, seq_env, last_row, d,
                       eps, h_pre, h_norm);
}

// ------------------------------------------------------- small linear --
// One wave per output column n, for all R input rows: the lanes read W's row
// n and each input row in coalesced 64-element strides, then sum across the
// wave (a fixed butterfly).
template <typename T>
__global__ __launch_bounds__(256) void small_linear_kernel(const float* in, int R, int K, const T* W, int N,
                                                           float* out, int silu_input)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = blockIdx.x * 4 + wave;
    if (n >= N) return;
    const T* w = W + (size_t)n * K;
    for (int r = 0; r < R; ++r) {
        const float* x = in + (size_t)r * K;
        float acc = 0.f;
        for (int k = lane; k < K; k += 64) {
            float v = x[k];
            if (silu_input) v = v / (1.0f + expf(-v));
            acc = fmaf(v, ld_elem<T>(w + k), acc);
        }
        acc = wave_sum(acc);
        if (lane == 0) out[(size_t)r * N + n] = acc;
    }
}

void small_linear(bool bf16, const float* in, int R, int K, const void* W, int N, float* out,
                  bool silu_input, hipStream_t s) {
    if (R <= 0 || N <= 0) return;
    const dim3 grid((N + 3) / 4);
    if (bf16)
        hipLaunchKernelGGL(small_linear_kernel<bf16_t>, grid, dim3(256), 0, s, in, R, K, (const bf16_t*)W, N,
                           out, (int)silu_input);
    else
        hipLaunchKernelGGL(small_linear_kernel<float>, grid, dim3(256), 0, s, in, R, K, (const float*)W, N, out,
                           (int)silu_input);
}

// ------------------------------------------------------------- flow --
// The denoised tokens of one env sit in `per_out` consecutive rows of H; a
// modality's token r (its rows numbered env by env, `per_in` per env) is
// H row (r / per_in) * per_out + off + r % per_in.  Actions alone: per_in =
// per_out = chunk, off = 0; the world-action model puts an env's future-frame
// latents first and its action tokens after them.
EBRL_DEV size_t flow_row(int r, int per_in, int per_out, int off) {
    return (size_t)(r / per_in) * per_out + off + r % per_in;
}

// A workgroup projects FLOW_IN_ROWS tokens onto 256 of the d outputs (grid:
// row blocks x output slices, so that even a few thousand tokens fill the
// chip): the tokens' inputs sit in LDS, each thread keeps its output's
// weight row in registers and runs four tokens at a time (independent FMA
// chains).  Each output is summed over the input channels in channel order,
// then the time embedding is added.
constexpr int FLOW_IN_ROWS = 16;
template <typename T, int AMAX>
__global__ __launch_bounds__(256) void flow_in_kernel(const float* __restrict__ x, int rows, int adim,
                                                      const T* __restrict__ W_ain, const float* __restrict__ tvec,
                                                      int d, float* __restrict__ H, int ldh, int per_in,
                                                      int per_out, int off)
{
    static_assert(FLOW_IN_ROWS % 4 == 0, "four tokens per pass");
    __shared__ float sx[FLOW_IN_ROWS * AMAX];
    const int r0 = blockIdx.x * FLOW_IN_ROWS;
    const int nr = min(FLOW_IN_ROWS, rows - r0);
    for (int i = threadIdx.x; i < FLOW_IN_ROWS * AMAX; i += blockDim.x) {
        const int q = i / AMAX, j = i - q * AMAX;
        sx[i] = (q < nr && j < adim) ? x[(size_t)(r0 + q) * adim + j] : 0.f;
    }
    __syncthreads();
    const int o = blockIdx.y * blockDim.x + threadIdx.x;
    if (o >= d) return;
    float w[AMAX];
#pragma unroll
    for (int j = 0; j < AMAX; ++j) w[j] = j < adim ? ld_elem<T>(W_ain + (size_t)o * adim + j) : 0.f;
    const float t = tvec[o];
    for (int q0 = 0; q0 < nr; q0 += 4) {
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < AMAX; ++j) {
            if (j < adim) {
#pragma unroll
                for (int u = 0; u < 4; ++u) acc[u] = fmaf(w[j], sx[(q0 + u) * AMAX + j], acc[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (q0 + u < nr) H[flow_row(r0 + q0 + u, per_in, per_out, off) * ldh + o] = acc[u] + t;
    }
}

void flow_in(bool bf16, const float* x, int rows, int adim, const void* W_ain, const float* tvec,
             int d, float* H, int ldh, int per_in, int per_out, int off, hipStream_t s) {
    if (rows <= 0) return;
    const dim3 grid((rows + FLOW_IN_ROWS - 1) / FLOW_IN_ROWS, (d + 255) / 256);
    auto go = [&](auto amax) {
        constexpr int AM = decltype(amax)::value;
        if (bf16)
            hipLaunchKernelGGL((flow_in_kernel<bf16_t, AM>), grid, dim3(256), 0, s, x, rows, adim,
                               (const bf16_t*)W_ain, tvec, d, H, ldh, per_in, per_out, off);
        else
            hipLaunchKernelGGL((flow_in_kernel<float, AM>), grid, dim3(256), 0, s, x, rows, adim,
                               (const float*)W_ain, tvec, d, H, ldh, per_in, per_out, off);
    };
    if (adim <= 8) go(std::integral_constant<int, 8>{});
    else if (adim <= 32) go(std::integral_constant<int, 32>{});
    else go(std::integral_constant<int, 64>{});   // adim <= 64 (checked at policy creation)
}

template <typename T>
__global__ __launch_bounds__(256) void flow_out_kernel(const float* H, int ldh, int d, const T* W_aout,
                                                       int adim, float eps, float n_steps, float* x,
                                                       float* v_out, int per_in, int per_out, int off)
{
    extern __shared__ float sh[];
    float* hn = sh;          // [d]
    float* vv = sh + d;      // [adim]
    __shared__ float red[16];
    const int r = blockIdx.x;
    const float* h = H + flow_row(r, per_in, per_out, off) * ldh;
    const float rs = row_rstd(h, d, eps, red);
    for (int j = threadIdx.x; j < d; j += blockDim.x) hn[j] = h[j] * rs;
    __syncthreads();
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
    for (int c = wave; c < adim; c += nw) {
        float dot = 0.f;
        for (int j = lane; j < d; j += 64) dot = fmaf(ld_elem<T>(W_aout + (size_t)c * d + j), hn[j], dot);
        dot = wave_sum(dot);
        if (lane == 0) vv[c] = dot;
    }
    __syncthreads();
    for (int c = threadIdx.x; c < adim; c += blockDim.x) {
        const float v = vv[c];
        x[(size_t)r * adim + c] -= v / n_steps;
        if (v_out) v_out[(size_t)r * adim + c] = v;
    }
}

// The same projection with RW rows per wave (four waves per workgroup):
// each lane holds columns 256 i + 4 lane .. + 3 of its rows in registers, a
// weight row is loaded once for all of them, and every dot product and
// sum of squares is summed per lane in column order, then over the lanes
// (wave_sum).  For d a multiple of 256 up to 2048.
template <typename T, int D4, int RW>
__global__ __launch_bounds__(256) void flow_out_rows_kernel(const float* __restrict__ H, int ldh, int d,
                                                            const T* __restrict__ W_aout, int adim, float eps,
                                                            float n_steps, float* __restrict__ x,
                                                            float* __restrict__ v_out, int rows, int per_in,
                                                            int per_out, int off)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int r0 = (blockIdx.x * 4 + wave) * RW;
    float4 hv[RW][D4];
#pragma unroll
    for (int k = 0; k < RW; ++k) {
        float ss = 0.f;
        if (r0 + k < rows) {
            const float* h = H + flow_row(r0 + k, per_in, per_out, off) * ldh + 4 * lane;
#pragma unroll
            for (int i = 0; i < D4; ++i) {
                hv[k][i] = *reinterpret_cast<const float4*>(h + 256 * i);
                ss = fmaf(hv[k][i].x, hv[k][i].x, ss);
                ss = fmaf(hv[k][i].y, hv[k][i].y, ss);
                ss = fmaf(hv[k][i].z, hv[k][i].z, ss);
                ss = fmaf(hv[k][i].w, hv[k][i].w, ss);
            }
        } else {
#pragma unroll
            for (int i = 0; i < D4; ++i) hv[k][i] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
        ss = wave_sum(ss);
        const float rs = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
        for (int i = 0; i < D4; ++i) {
            hv[k][i].x *= rs; hv[k][i].y *= rs; hv[k][i].z *= rs; hv[k][i].w *= rs;
        }
    }
    float mine[RW];
#pragma unroll
    for (int k = 0; k < RW; ++k) mine[k] = 0.f;
    for (int c = 0; c < adim; ++c) {
        const T* wr = W_aout + (size_t)c * d + 4 * lane;
        float acc[RW];
#pragma unroll
        for (int k = 0; k < RW; ++k) acc[k] = 0.f;
#pragma unroll
        for (int i = 0; i < D4; ++i) {
            float w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = ld_elem<T>(wr + 256 * i + e);
#pragma unroll
            for (int k = 0; k < RW; ++k) {
                acc[k] = fmaf(w[0], hv[k][i].x, acc[k]);
                acc[k] = fmaf(w[1], hv[k][i].y, acc[k]);
                acc[k] = fmaf(w[2], hv[k][i].z, acc[k]);
                acc[k] = fmaf(w[3], hv[k][i].w, acc[k]);
            }
        }
#pragma unroll
        for (int k = 0; k < RW; ++k) {
            const float v = wave_sum(acc[k]);
            if (lane == c) mine[k] = v;
        }
    }
#pragma unroll
    for (int k = 0; k < RW; ++k) {
        const int r = r0 + k;
        if (r < rows && lane < adim) {
            x[(size_t)r * adim + lane] -= mine[k] / n_steps;
            if (v_out) v_out[(size_t)r * adim + lane] = mine[k];
        }
    }
}

void flow_out(bool bf16, const float* H, int ldh, int rows, int d, const void* W_aout, int adim,
              float eps, float n_steps, float* x, float* v_out, int per_in, int per_out, int off,
              hipStream_t s) {
    if (rows <= 0) return;
    auto go = [&](auto d4, auto rw) {
        constexpr int D4 = decltype(d4)::value, RW = decltype(rw)::value;
        const dim3 grid((rows + 4 * RW - 1) / (4 * RW));
        if (bf16)
            hipLaunchKernelGGL((flow_out_rows_kernel<bf16_t, D4, RW>), grid, dim3(256), 0, s, H, ldh, d,
                               (const bf16_t*)W_aout, adim, eps, n_steps, x, v_out, rows, per_in, per_out, off);
        else
            hipLaunchKernelGGL((flow_out_rows_kernel<float, D4, RW>), grid, dim3(256), 0, s, H, ldh, d,
                               (const float*)W_aout, adim, eps, n_steps, x, v_out, rows, per_in, per_out, off);
    };
    using std::integral_constant;
    if (d % 256 == 0 && adim <= 64) {
        switch (d / 256) {
        case 1: go(integral_constant<int, 1>{}, integral_constant<int, 4>{}); return;
        case 2: go(integral_constant<int, 2>{}, integral_constant<int, 4>{}); return;
        case 3: go(integral_constant<int, 3>{}, integral_constant<int, 4>{}); return;
        case 4: go(integral_constant<int, 4>{}, integral_constant<int, 4>{}); return;
        case 6: go(integral_constant<int, 6>{}, integral_constant<int, 2>{}); return;
        case 8: go(integral_constant<int, 8>{}, integral_constant<int, 2>{}); return;
        default: break;
        }
    }
    const size_t shm = (size_t)(d + adim) * sizeof(float);
    if (bf16)
        hipLaunchKernelGGL(flow_out_kernel<bf16_t>, dim3(rows), dim3(256), shm, s, H, ldh, d,
                           (const bf16_t*)W_aout, adim, eps, n_steps, x, v_out, per_in, per_out, off);
    else
        hipLaunchKernelGGL(flow_out_kernel<float>, dim3(rows), dim3(256), shm, s, H, ldh, d,
                           (const float*)W_aout, adim, eps, n_steps, x, v_out, per_in, per_out, off);
}

__global__ void copy_f32_kernel(const float* src, float* dst, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

void copy_f32(const float* src, float* dst, size_t n, hipStream_t s) {
    if (n == 0) return;
    const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(copy_f32_kernel, dim3(blocks), dim3(256), 0, s, src, dst, n);
}

__global__ void copy_decode_out_kernel(const int* tok, const float* act, const float* mar, int count, int* out_tok,
                                       float* out_act, float* out_mar) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < count; i += gridDim.x * blockDim.x) {
        out_tok[i] = tok[i];
        if (out_act) out_act[i] = act[i];
        if (out_mar) out_mar[i] = mar[i];
    }
}

void copy_decode_out(const int* tok, const float* act, const float* mar, int count, int* out_tok, float* out_act,
                     float* out_mar, hipStream_t s) {
    if (count <= 0) return;
    const int blocks = std::min((count + 255) / 256, 1024);
    hipLaunchKernelGGL(copy_decode_out_kernel, dim3(blocks), dim3(256), 0, s, tok, act, mar, count, out_tok, out_act,
                       out_mar);
}


// ---------------------------------------------------------- seeded noise --
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), ten rounds of
//   (c0, c1, c2, c3) <- (mulhi(B, c2) ^ c1 ^ k0, mullo(B, c2),
//                        mulhi(A, c0) ^ c3 ^ k1, mullo(A, c0)),
// A = 0xD2511F53, B = 0xCD9E8D57, key bumped by (0x9E3779B9, 0xBB67AE85)
// before every round but the first; then Box-Muller (1958) on the first two
// words, u = (x + 1/2) 2^-32, in double, rounded to float.  Row i's pair j
// takes counter (j, calls[i], env[i], stream) under key (lo, hi of seed).
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint32_t hb = __umulhi(0xCD9E8D57u, c[2]), lb = 0xCD9E8D57u * c[2];
        const uint32_t ha = __umulhi(0xD2511F53u, c[0]), la = 0xD2511F53u * c[0];
        const uint32_t n0 = hb ^ c[1] ^ k0, n2 = ha ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lb;
        c[2] = n2;
        c[3] = la;
    }
}

__global__ __launch_bounds__(256) void normal_noise_kernel(float* __restrict__ out, int per_row,
                                                           const int* __restrict__ env,
                                                           const int* __restrict__ calls, uint32_t k0,
                                                           uint32_t k1, uint32_t stream) {
    const int i = blockIdx.y;
    const int pairs = (per_row + 1) / 2;
    const uint32_t e = (uint32_t)env[i], call = (uint32_t)calls[i];
    for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < pairs; j += gridDim.x * blockDim.x) {
        uint32_t c[4] = {(uint32_t)j, call, e, stream};
        philox4x32_10(c, k0, k1);
        const double u1 = ((double)c[0] + 0.5) * (1.0 / 4294967296.0);
        const double u2 = ((double)c[1] + 0.5) * (1.0 / 4294967296.0);
        const double rad = sqrt(-2.0 * log(u1));
        const double ang = 6.283185307179586 * u2;
        float* o = out + (size_t)i * per_row + 2 * j;
        o[0] = (float)(rad * cos(ang));
        if (2 * j + 1 < per_row) o[1] = (float)(rad * sin(ang));
    }
}

void normal_noise(float* out, int rows, int per_row, const int* env, const int* calls, uint64_t seed,
                  uint32_t stream, hipStream_t s) {
    if (rows <= 0 || per_row <= 0) return;
    const int pairs = (per_row + 1) / 2;
    dim3 grid((unsigned)std::min((pairs + 255) / 256, 64), (unsigned)rows);
    hipLaunchKernelGGL(normal_noise_kernel, grid, dim3(256), 0, s, out, per_row, env, calls,
                       (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32), stream);
}


// ------------------------------------------------------- streaming read --
// Workgroup b reads 16-byte words [b * per, (b + 1) * per) with eight
// non-temporal loads in flight per lane.  A lane writes *out only if the XOR
// of its words equals a fixed constant, so every load's value is used.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ p, size_t n16, size_t per,
                                                          unsigned* out)
{
    constexpr int U = 8;
    u32x4 acc = {0u, 0u, 0u, 0u};
    const size_t b0 = blockIdx.x * per, b1 = min(n16, b0 + per);
    for (size_t i = b0 + threadIdx.x; i < b1; i += 256 * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t j = i + (size_t)u * 256;
            v[u] = j < b1 ? __builtin_nontemporal_load(p + j) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u];
    }
    const unsigned x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    if (x == 0x9E3779B9u) *out = x;
}

void stream_read(const void* buf, size_t bytes, unsigned* out, hipStream_t s) {
    const size_t n16 = bytes / 16;
    const int grid = 4096;
    const size_t per = (n16 + grid - 1) / grid;
    hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(256), 0, s, (const u32x4*)buf, n16, per, out);
}

}  // namespace ebrl
