// Softmax attention softmax(Q K^T / sqrt(hd) + mask) V over the paged KV
// cache (16-token blocks), for every query head h reading KV head
// h / (q_heads / kv_heads).
//
// attn_prefill_bf16: flash attention for prefill, the ViT and the flow
//   expert.  A workgroup (4 waves) owns 64 query rows of one head; K and V
//   tiles (32 keys at hd 128, 64 at hd 64) are DMA'd from the paged cache
//   into double-buffered LDS
//   (whole 128/256-byte rows, XOR-swizzled 16-byte chunks).  Each wave
//   computes S^T = K Q^T for its 16 queries with v_mfma_f32_16x16x32_bf16 so
//   that every lane holds the scores of a single query, runs the online
//   softmax in fp32 with exp2, and feeds the probabilities straight back as
//   the B operand of O^T = V^T P^T; V stays row-major in LDS and the
//   transposed fragments come from ds_read_b64_tr_b16.  P enters the bf16
//   product as 2^(x - ceil(max x)), x = s log2(e) / sqrt(hd), with the row
//   sum taken before rounding.
// attn_prefill_f32: plain per-(query, head) kernel for fp32 policies.
// attn_decode_bf16: one query per sequence; one workgroup per (sequence,
//   head, chunk of keys) with whole-row loads, chunks merged in chunk order
//   by the last workgroup of a (sequence, head).  attn_decode_split (+
//   combine): the fp32 path, 64-key chunks merged by a second kernel in
//   chunk order.
#include <math.h>

#include <type_traits>

#include "kernels.h"

namespace ebrl {

// --------------------------------------------------------- bf16 prefill --

typedef __attribute__((address_space(3))) void* attn_lds_ptr_t;
typedef short attn_v4s __attribute__((ext_vector_type(4)));

// global_load_lds_dwordx4 issued as inline assembly: the compiler neither
// counts it nor guards LDS reads against it; the kernel waits on vmcnt and
// synchronises the workgroup itself before reading a filled buffer.
EBRL_DEV void attn_dma16(const void* g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(g), "s"(lds_addr) : "memory", "m0");
}

// Lanes l and l ^ 16, then l and l ^ 32, combined with VALU lane swaps
// (v_permlane16_swap / v_permlane32_swap hand each lane both values of its
// pair), instead of LDS-routed swizzles that queue behind the K/V traffic.
// Both lanes of a pair get the same result (the operations commute).
EBRL_DEV float attn_max_xor16_32(float v) {
    const unsigned u = __builtin_bit_cast(unsigned, v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = fmaxf(__builtin_bit_cast(float, (unsigned)a[0]), __builtin_bit_cast(float, (unsigned)a[1]));
    const unsigned w = __builtin_bit_cast(unsigned, v);
    const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
    return fmaxf(__builtin_bit_cast(float, (unsigned)b[0]), __builtin_bit_cast(float, (unsigned)b[1]));
}
EBRL_DEV float attn_sum_xor16_32(float v) {
    const unsigned u = __builtin_bit_cast(unsigned, v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = __builtin_bit_cast(float, (unsigned)a[0]) + __builtin_bit_cast(float, (unsigned)a[1]);
    const unsigned w = __builtin_bit_cast(unsigned, v);
    const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
    return __builtin_bit_cast(float, (unsigned)b[0]) + __builtin_bit_cast(float, (unsigned)b[1]);
}

// One KT-key tile (a multiple of 32) of the online-softmax attention for the
// wave's 16 queries (lane (r, g): query r, keys 16 kt + 4 g + v): scores
// S^T = K Q^T on MFMA, masking, the integer running maximum, P, and
// O^T += V^T P^T.  tk / tv point at the tile's K and V rows in LDS (KT rows
// of HD, 16-byte chunks swizzled by row).
template <int HD, int KT>
EBRL_DEV void attn_tile_math(const bf16_t* tk, const bf16_t* tv, int k0, int mask_from, int key_lim,
                             float scale_log2, const bf16x8 (&qb)[HD / 32], float& m_i, float& l_i,
                             f32x4 (&acc)[HD / 16], int lane)
{
    static_assert(KT % 32 == 0, "whole 32-key MFMA steps");
    constexpr int NKT = KT / 16, CPR = HD / 8;
    const int r = lane & 15, g = lane >> 4;
    // S^T tiles: lane holds key 16kt + 4g + v for query r
    f32x4 s[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
        s[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int row = kt * 16 + r;
#pragma unroll
        for (int ks = 0; ks < HD / 32; ++ks) {
            const bf16x8 ka =
                *reinterpret_cast<const bf16x8*>(tk + (row * CPR + ((ks * 4 + g) ^ (row & (CPR - 1)))) * 8);
            s[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qb[ks], s[kt], 0, 0, 0);
        }
    }
    // Row maximum of the raw scores: the scale is positive, so it
    // commutes with the maximum and is applied once, inside the
    // exponent's fused multiply-add.  Masked scores become -inf.
    if (mask_from <= k0 + KT - 1) {
        // tile reaches past the keys or past a query of this wave: key
        // k0 + 16 kt + 4 g + v is visible to this lane's query iff
        // 16 kt + v < lim
        const int lim = key_lim - k0 - 4 * g;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
            for (int v = 0; v < 4; ++v) s[kt][v] = kt * 16 + v < lim ? s[kt][v] : -INFINITY;
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) tmax = fmaxf(tmax, s[kt][v]);
    tmax = attn_max_xor16_32(tmax);
    // The running maximum is kept as an integer (ceil, in log2 units):
    // rescaling by alpha is then a power of two, which commutes with the
    // bf16 rounding of P, so P is rounded as 2^(x - ceil(row max)) no
    // matter how the keys are split into tiles.
    const float m_new = fmaxf(m_i, ceilf(tmax * scale_log2));
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = (m_i == -INFINITY) ? 0.f : ldexpf(1.0f, (int)(m_i - m_use));
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float p = fast_exp2(fmaf(s[kt][v], scale_log2, -m_use));
            s[kt][v] = p;
            psum += p;
        }
    psum = attn_sum_xor16_32(psum);
    l_i = l_i * alpha + psum;
    m_i = m_new;
    // alpha is a power of two (1 once the integer running maximum stops
    // growing), so the rescale is exact; it is applied unconditionally, which
    // keeps the accumulators in place (a branch around it costs register
    // copies on both paths)
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) acc[i] *= alpha;

    // O^T += V^T P^T.  V stays row-major in LDS; ds_read_b64_tr_b16 hands
    // lane (r, g) the values of dimension 16 dt + r for 4 keys per read
    // (keys 32 ks2 + 4g + j, then 32 ks2 + 16 + 4g + j), the same key
    // order the score lanes hold.
    const int a16 = lane & 15;
#pragma unroll
    for (int ks2 = 0; ks2 < KT / 32; ++ks2) {
        bf16x8 pb;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            pb[v] = (__bf16)s[2 * ks2][v];
            pb[4 + v] = (__bf16)s[2 * ks2 + 1][v];
        }
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) {
            const int d = dt * 16 + 4 * (a16 & 3);
            attn_v4s lo, hi;
            {
                const int key = 32 * ks2 + 4 * g + (a16 >> 2);
                const int off = (key * CPR + ((d >> 3) ^ (key & (CPR - 1)))) * 8 + (d & 7);
                lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) attn_v4s*)(attn_lds_ptr_t)(tv + off));
            }
            {
                const int key = 32 * ks2 + 16 + 4 * g + (a16 >> 2);
                const int off = (key * CPR + ((d >> 3) ^ (key & (CPR - 1)))) * 8 + (d & 7);
                hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) attn_v4s*)(attn_lds_ptr_t)(tv + off));
            }
            const uint2 lo2 = __builtin_bit_cast(uint2, lo), hi2 = __builtin_bit_cast(uint2, hi);
            const uint4 w = make_uint4(lo2.x, lo2.y, hi2.x, hi2.y);
            const bf16x8 va = __builtin_bit_cast(bf16x8, w);
            acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, acc[dt], 0, 0, 0);
        }
    }
}

// s_waitcnt on the vector-memory counter only (gfx9 encoding: expcnt and
// lgkmcnt fields at their maxima).
template <int N> EBRL_DEV void attn_wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | 0xF00 | ((N >> 4) << 14));
}

// One workgroup per (query tile of ATTN_Q_TILE rows, head): NW waves of 16
// queries share every K/V tile staged in LDS, which each wave then skips if
// none of its queries can see it.  Key tiles of KT keys in an S-buffer ring:
// S - 1 tiles are in flight while one is multiplied.
template <int HD, int NW, int KT, int S>
__global__ __launch_bounds__(64 * NW) void attn_prefill_bf16_kernel(AttnPrefillArgs a, float scale_log2)
{
    static_assert(16 * NW == ATTN_Q_TILE, "query tile");
    static_assert(S >= 2 && S <= 4, "ring depth");
    constexpr int CPR = HD / 8;            // 16-byte chunks per K/V row
    constexpr int RPI = 64 / CPR;          // rows per DMA instruction
    constexpr int TILE = KT * HD;          // bf16 per K (or V) tile
    __shared__ __attribute__((aligned(1024))) bf16_t sK[S][TILE];
    __shared__ __attribute__((aligned(1024))) bf16_t sV[S][TILE];
    __shared__ int s_bt[ATTN_BT_MAX];

    // Workgroup order: the dispatcher deals workgroup ids round-robin over
    // the 8 XCDs, each with its own L2.  Ids are remapped so that every XCD
    // runs a contiguous run of (KV head, query tile, query head in the KV
    // group) triples: the query heads of one KV group and the query tiles of
    // one sequence, which read the same K and V, share an L2 (the world
    // action model's attention: 15 % faster).  Causal attention without
    // grouped heads keeps the dispatcher's order, which measured 3 % faster
    // there.
    const int hkv = a.kv.kv_heads;
    const int grp = a.q_heads / hkv;
    int lid = blockIdx.x;
    const int nb = gridDim.x;
    if ((nb & 7) == 0 && (!a.causal || grp > 1)) lid = (lid & 7) * (nb >> 3) + (lid >> 3);
    const int rest = lid / grp;
    const int t = rest % a.n_tiles, kvh = rest / a.n_tiles;
    const int h = kvh * grp + (lid - rest * grp);
    const int seq = a.tile_seq[t], qt0 = a.tile_q0[t];
    const int env = a.seq_env[seq];
    const int qlen = a.q_len[seq], qpos0 = a.q_pos0[seq], kvlen = a.kv_len[seq];
    const int qoff = a.q_off[seq];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int qi = qt0 + wave * 16 + r;
    const bool qvalid = qi < qlen;
    const int qpos = qpos0 + qi;

    int kv_end = kvlen;
    if (a.causal) kv_end = min(kvlen, qpos0 + min(qt0 + ATTN_Q_TILE, qlen));
    // first key that some lane of this wave must mask: the end of the keys, or
    // (causal) the position of the wave's first query plus one
    const int mask_from = a.causal ? min(kvlen, qpos0 + qt0 + wave * 16 + 1) : kvlen;
    // one past the last key this lane's query may see
    const int key_lim = a.causal ? min(kvlen, qpos + 1) : kvlen;
    // the last key any query of this wave may see (none: the wave idles)
    const int wq0 = qt0 + wave * 16;
    const int wave_keys = wq0 >= qlen ? 0 : (a.causal ? min(kvlen, qpos0 + min(wq0 + 16, qlen)) : kvlen);
    const int ntiles = (kv_end + KT - 1) / KT;
    for (int b2 = tid; b2 < (kv_end + KV_BLOCK - 1) / KV_BLOCK; b2 += 64 * NW)
        s_bt[b2] = a.kv.block_table[(size_t)env * a.kv.bt_stride + b2];

    bf16x8 qb[HD / 32];
    {
        const bf16_t* qrow = (const bf16_t*)a.Q + (size_t)(qoff + min(qi, qlen - 1)) * a.ldq + h * HD;
#pragma unroll
        for (int ks = 0; ks < HD / 32; ++ks) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (qvalid) v = *reinterpret_cast<const uint4*>(qrow + ks * 32 + g * 8);
            qb[ks] = *reinterpret_cast<bf16x8*>(&v);
        }
    }
    __syncthreads();

    // DMA of key tile `it`: row q of the tile = key k0 + q, its 16-byte chunk
    // c stored at chunk position q * CPR + (c ^ (q % CPR)) -- the XOR spans
    // every chunk of a row, so that 8 (hd 64) or 16 (hd 128) consecutive rows
    // put a given chunk on all 64 LDS banks; the waves split the
    // tile's KT / RPI instructions for K and the same for V, so that wave w
    // fills rows RW w .. RW w + RW - 1, which lie in one 16-token cache block.
    constexpr int RW = KT / NW;              // rows per wave
    static_assert((KT / RPI) % NW == 0, "DMA split");
    static_assert(KV_BLOCK == 16 && 16 % RW == 0 && KT % 16 == 0, "a wave's rows in one cache block");
    constexpr int NI = KT / RPI;             // instructions per operand
    constexpr int IPT = 2 * (NI / NW);       // DMA instructions per tile and wave (K and V)
    const size_t blk_elems = (size_t)2 * hkv * KV_BLOCK * HD;
    const bf16_t* kbase = (const bf16_t*)a.kv.base + (size_t)kvh * KV_BLOCK * HD;
    const size_t voff = (size_t)hkv * KV_BLOCK * HD;
    const uint32_t sk_addr = (uint32_t)(uintptr_t)(attn_lds_ptr_t)&sK[0][0];
    const uint32_t sv_addr = (uint32_t)(uintptr_t)(attn_lds_ptr_t)&sV[0][0];
    const int row_in = lane / CPR, cpos = lane % CPR;
    auto dma = [&](int it, int buf) {
        const int blk_key0 = it * KT + wave * RW;     // first key of this wave's rows
        if (blk_key0 + RW <= kv_end) {
            // whole block in range: its address is uniform over the wave
            const int blk = __builtin_amdgcn_readfirstlane(s_bt[blk_key0 >> 4]);
            const bf16_t* kb = kbase + (size_t)blk * blk_elems;
#pragma unroll
            for (int u = 0; u < NI / NW; ++u) {
                const int ins = wave * (NI / NW) + u;
                const int q = ins * RPI + row_in;
                const int c = cpos ^ (q & (CPR - 1));
                const bf16_t* src = kb + (size_t)(((it * KT + q) & 15) * HD + c * 8);
                const uint32_t off = (uint32_t)(buf * TILE + ins * 512) * 2;
                attn_dma16(src, __builtin_amdgcn_readfirstlane(sk_addr + off));
                attn_dma16(src + voff, __builtin_amdgcn_readfirstlane(sv_addr + off));
            }
        } else {
            // the block holding the last keys: rows past them repeat the
            // last key (finite values; their scores are masked)
#pragma unroll
            for (int u = 0; u < NI / NW; ++u) {
                const int ins = wave * (NI / NW) + u;
                const int q = ins * RPI + row_in;
                const int key = min(it * KT + q, kv_end - 1);
                const int c = cpos ^ (q & (CPR - 1));
                const bf16_t* src = kbase + (size_t)s_bt[key >> 4] * blk_elems + (size_t)(key & 15) * HD + c * 8;
                const uint32_t off = (uint32_t)(buf * TILE + ins * 512) * 2;
                attn_dma16(src, __builtin_amdgcn_readfirstlane(sk_addr + off));
                attn_dma16(src + voff, __builtin_amdgcn_readfirstlane(sv_addr + off));
            }
        }
    };

    f32x4 acc[HD / 16];
#pragma unroll
    for (int i = 0; i < HD / 16; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_i = -INFINITY, l_i = 0.f;

    // One key tile from LDS buffer BUF (a compile-time constant, so that
    // every fragment address is a per-lane base plus an immediate offset).
    auto tile = [&](int it, auto BUF) {
        constexpr int buf = decltype(BUF)::value;
        // this wave's part of tile `it` has landed (the tiles issued after it
        // may stay in flight); after the barrier every wave's part has, and
        // every wave is done with tile it - 1, whose buffer the next DMA refills
        const int later = min(S - 2, ntiles - 1 - it);
        if (later >= 2) attn_wait_vmcnt<2 * IPT>();
        else if (later == 1) attn_wait_vmcnt<IPT>();
        else attn_wait_vmcnt<0>();
        __syncthreads();
        if (it + S - 1 < ntiles) dma(it + S - 1, (buf + S - 1) % S);
        const bf16_t* tk = sK[buf];
        const bf16_t* tv = sV[buf];
        const int k0 = it * KT;
        // no query of this wave sees a key of this tile: nothing to add
        // (processing it would leave m, l and acc as they are)
        if (k0 >= wave_keys) return;

        attn_tile_math<HD, KT>(tk, tv, k0, mask_from, key_lim, scale_log2, qb, m_i, l_i, acc, lane);
    };

    for (int p = 0; p < S - 1 && p < ntiles; ++p) dma(p, p);
    for (int it = 0; it < ntiles; it += S) {
        tile(it, std::integral_constant<int, 0>{});
        if (it + 1 < ntiles) tile(it + 1, std::integral_constant<int, 1>{});
        if constexpr (S > 2) {
            if (it + 2 < ntiles) tile(it + 2, std::integral_constant<int, 2 % S>{});
        }
        if constexpr (S > 3) {
            if (it + 3 < ntiles) tile(it + 3, std::integral_constant<int, 3 % S>{});
        }
    }

    if (qvalid) {
        const float inv = l_i > 0.f ? 1.f / l_i : 0.f;
        bf16_t* orow = (bf16_t*)a.O + (size_t)(qoff + qi) * a.ldo + h * HD;
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt)
            st4<bf16_t>(orow + dt * 16 + 4 * g, acc[dt][0] * inv, acc[dt][1] * inv,
                        acc[dt][2] * inv, acc[dt][3] * inv);
    }
}

// ---------------------------------------------------------- fp32 prefill --
// grid (tile, head, ATTN_Q_TILE rows of the tile); one wave per query row.
__global__ __launch_bounds__(64) void attn_prefill_f32_kernel(AttnPrefillArgs a, float scale)
{
    extern __shared__ float sh[];
    const int t = blockIdx.x, h = blockIdx.y;
    const int seq = a.tile_seq[t];
    const int qi = a.tile_q0[t] + blockIdx.z;
    const int qlen = a.q_len[seq];
    if (qi >= qlen) return;
    const int env = a.seq_env[seq];
    const int hd = a.kv.head_dim, hkv = a.kv.kv_heads;
    const int kvh = h / (a.q_heads / hkv);
    const int qpos = a.q_pos0[seq] + qi;
    int kvlen = a.kv_len[seq];
    if (a.causal) kvlen = min(kvlen, qpos + 1);
    float* q = sh;          // [hd]
    float* sc = sh + hd;    // [kvlen]
    const float* qrow = (const float*)a.Q + (size_t)(a.q_off[seq] + qi) * a.ldq + h * hd;
    const int lane = threadIdx.x;
    for (int i = lane; i < hd; i += 64) q[i] = qrow[i];
    __syncthreads();
    const size_t blk_elems = (size_t)2 * hkv * KV_BLOCK * hd;
    const float* base = (const float*)a.kv.base;
    const int* bt = a.kv.block_table + (size_t)env * a.kv.bt_stride;
    float mx = -INFINITY;
    for (int j = lane; j < kvlen; j += 64) {
        const float* kr = base + (size_t)bt[j >> 4] * blk_elems + ((size_t)kvh * KV_BLOCK + (j & 15)) * hd;
        float dot = 0.f;
        for (int i = 0; i < hd; ++i) dot = fmaf(q[i], kr[i], dot);
        dot *= scale;
        sc[j] = dot;
        mx = fmaxf(mx, dot);
    }
    mx = wave_max(mx);
    float sum = 0.f;
    for (int j = lane; j < kvlen; j += 64) {
        const float p = expf(sc[j] - mx);
        sc[j] = p;
        sum += p;
    }
    sum = wave_sum(sum);
    __syncthreads();
    float* orow = (float*)a.O + (size_t)(a.q_off[seq] + qi) * a.ldo + h * hd;
    for (int i = lane; i < hd; i += 64) {
        float o = 0.f;
        for (int j = 0; j < kvlen; ++j) {
            const float* vr = base + (size_t)bt[j >> 4] * blk_elems +
                              ((size_t)(hkv + kvh) * KV_BLOCK + (j & 15)) * hd;
            o = fmaf(sc[j], vr[i], o);
        }
        orow[i] = o / sum;
    }
}

void attn_prefill(const AttnPrefillArgs& a, hipStream_t s) {
    if (a.n_tiles <= 0) return;
    const int hd = a.kv.head_dim;
    if (a.bf16) {
        if (a.kv.bt_stride > ATTN_BT_MAX) return;   // rejected by the caller (capacity check)
        const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
        dim3 grid(a.n_tiles * a.q_heads);
        constexpr int NW = ATTN_Q_TILE / 16;
        // hd 128: 32-key tiles (32 KB of LDS: up to four workgroups per CU)
        // measured 9-15 % faster than 64-key tiles; hd 64 keeps 64-key tiles
        // (32-key ones 3 % slower).  Deeper rings (three 64-key or four 32-key
        // buffers) were slower at both widths.
        if (hd == 64) hipLaunchKernelGGL((attn_prefill_bf16_kernel<64, NW, 64, 2>), grid, dim3(64 * NW), 0, s, a, scale_log2);
        else hipLaunchKernelGGL((attn_prefill_bf16_kernel<128, NW, 32, 2>), grid, dim3(64 * NW), 0, s, a, scale_log2);
    } else {
        const float scale = 1.0f / sqrtf((float)hd);
        dim3 grid(a.n_tiles, a.q_heads, ATTN_Q_TILE);
        const size_t shm = (size_t)(hd + a.max_kv_len) * sizeof(float);
        hipLaunchKernelGGL(attn_prefill_f32_kernel, grid, dim3(64), shm, s, a, scale);
    }
}

// ---------------------------------------------------------------- decode --

template <typename T> EBRL_DEV void load8(const T* p, float* o);
template <> EBRL_DEV void load8<bf16_t>(const bf16_t* p, float* o) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        o[2 * i] = __uint_as_float(w[i] << 16);
        o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}
template <> EBRL_DEV void load8<float>(const float* p, float* o) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}

// grid (n, q_heads, max_splits), 256 threads
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_decode_split_kernel(AttnDecodeArgs a, float scale_log2)
{
    constexpr int CH = ATTN_DEC_CHUNK;
    constexpr int LPK = HD / 8;          // lanes per key row
    constexpr int KPP = 256 / LPK;       // keys per pass
    __shared__ float sq[HD];
    __shared__ float ss[CH];
    __shared__ float sacc[KPP * HD];
    __shared__ float sml[2];

    const int i = blockIdx.x, h = blockIdx.y, sp = blockIdx.z;
    const int kvlen = a.kv_len[i];
    const int k0 = sp * CH;
    if (k0 >= kvlen) return;
    const int k1 = min(k0 + CH, kvlen);
    const int nkeys = k1 - k0;
    const int env = a.seq_env[i];
    const int hkv = a.kv.kv_heads;
    const int kvh = h / (a.q_heads / hkv);
    const int tid = threadIdx.x;
    const T* qrow = (const T*)a.Q + (size_t)i * a.ldq + h * HD;
    for (int d = tid; d < HD; d += 256) sq[d] = ld_elem<T>(qrow + d);
    __syncthreads();

    const size_t blk_elems = (size_t)2 * hkv * KV_BLOCK * HD;
    const T* base = (const T*)a.kv.base;
    const int* bt = a.kv.block_table + (size_t)env * a.kv.bt_stride;
    const int sub = tid % LPK, kg = tid / LPK;
    const int dc = sub * 8;

    for (int kk = kg; kk < CH; kk += KPP) {
        const int kidx = k0 + kk;
        float dot = 0.f;
        if (kk < nkeys) {
            const T* kr = base + (size_t)bt[kidx >> 4] * blk_elems +
                          ((size_t)kvh * KV_BLOCK + (kidx & 15)) * HD + dc;
            float kv[8];
            load8<T>(kr, kv);
#pragma unroll
            for (int j = 0; j < 8; ++j) dot = fmaf(sq[dc + j], kv[j], dot);
        }
#pragma unroll
        for (int off = LPK / 2; off > 0; off >>= 1) dot += __shfl_xor(dot, off, 64);
        if (sub == 0) ss[kk] = (kk < nkeys) ? dot * scale_log2 : -INFINITY;
    }
    __syncthreads();
    if (tid < 64) {
        const float v = ss[tid];
        const float m = wave_max(v);
        const float p = (tid < nkeys) ? fast_exp2(v - m) : 0.f;
        const float l = wave_sum(p);
        ss[tid] = p;
        if (tid == 0) { sml[0] = m; sml[1] = l; }
    }
    __syncthreads();
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    for (int kk = kg; kk < nkeys; kk += KPP) {
        const int kidx = k0 + kk;
        const T* vr = base + (size_t)bt[kidx >> 4] * blk_elems +
                      ((size_t)(hkv + kvh) * KV_BLOCK + (kidx & 15)) * HD + dc;
        float vv[8];
        load8<T>(vr, vv);
        const float p = ss[kk];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = fmaf(p, vv[j], acc[j]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) sacc[kg * HD + dc + j] = acc[j];
    __syncthreads();
    float* part = a.part + (((size_t)i * a.q_heads + h) * a.max_splits + sp) * (HD + 2);
    for (int d = tid; d < HD; d += 256) {
        float o = 0.f;
        for (int q = 0; q < KPP; ++q) o += sacc[q * HD + d];
        part[d] = o;
    }
    if (tid == 0) { part[HD] = sml[0]; part[HD + 1] = sml[1]; }
}

// bf16 decode attention.  A sequence of kv_len keys is cut into
// nch = ceil(kv_len / attn_decode_chunk(HD)) chunks of equal length (the last
// shorter), a function of its length only; one workgroup per (sequence,
// query head, chunk).  Its four waves take consecutive quarters of the chunk;
// a wave loads 8 K rows and the matching 8 V rows per lane per round in one
// burst (a load instruction covers whole 128-byte row segments: 8 keys of 64
// dims or 4 keys of 128) with non-temporal loads, keeps a running max / sum /
// weighted V, and the waves' states merge through LDS in wave order.  A
// one-chunk sequence writes its output there; with more chunks every
// workgroup stores its chunk state, and the workgroup that finishes a
// (sequence, head) last (a device-scope counter, left at zero again) merges
// the chunks in chunk order.  A sequence's bits therefore depend on its
// length only -- not on the batch, the grid or the order in which workgroups
// finish.  Chunks are long (512 keys at head dim 128): measured on the
// 7B-class decode, 128-key chunks (three to twelve times the workgroups, one
// load round each) streamed the cache 16 % slower than whole-sequence
// workgroups, the per-workgroup latency chain (block table, K/V, merge)
// outweighing the added parallelism; the split serves long sequences.

// 16-byte load marked non-temporal: each K/V row is read once per decode
// step, and streaming loads keep it from displacing cached data (measured:
// about 15 % more bandwidth than plain loads on the paged cache).
EBRL_DEV uint4 ld_stream16(const bf16_t* p) {
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

template <int HD> constexpr int attn_decode_chunk() { return 65536 / HD; }

template <int HD>
__global__ __launch_bounds__(256) void attn_decode_bf16_kernel(AttnDecodeArgs a, float scale_log2)
{
    constexpr int LPK = HD / 8;        // lanes per key row, 16 bytes each
    constexpr int KPL = 64 / LPK;      // keys per wave load
    constexpr int NL = 8;              // K (and V) loads per lane per round
    constexpr int KW = KPL * NL;       // keys per round
    constexpr int CK = attn_decode_chunk<HD>();
    constexpr int CB = CK / KV_BLOCK;  // cache blocks per chunk
    __shared__ int s_bt[CB + 1];       // a chunk may start inside a block
    __shared__ float s_o[4][HD];
    __shared__ float s_ml[4][2];
    __shared__ int s_last;

    const int i = blockIdx.x, h = blockIdx.y, c = blockIdx.z;
    const int kvlen = a.kv_len[i];
    const int nch = max(1, (kvlen + CK - 1) / CK);
    if (c >= nch) return;              // the grid covers the longest sequence
    const int clen = (kvlen + nch - 1) / nch;
    const int c0 = min(kvlen, c * clen), c1 = min(kvlen, c0 + clen);
    const int env = a.seq_env[i];
    const int hkv = a.kv.kv_heads;
    const int kvh = h / (a.q_heads / hkv);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int sub = lane % LPK, kq = lane / LPK;
    const int b0 = c0 >> 4;
    for (int b = tid; b < ((c1 + KV_BLOCK - 1) >> 4) - b0; b += 256)
        s_bt[b] = a.kv.block_table[(size_t)env * a.kv.bt_stride + b0 + b];
    float q[8];
    load8<bf16_t>((const bf16_t*)a.Q + (size_t)i * a.ldq + h * HD + sub * 8, q);
    __syncthreads();

    const int per = (c1 - c0 + 3) / 4;
    const int wb = min(c1, c0 + wave * per), we = min(c1, wb + per);
    const size_t blk_elems = (size_t)2 * hkv * KV_BLOCK * HD;
    const bf16_t* kbase = (const bf16_t*)a.kv.base + (size_t)kvh * KV_BLOCK * HD + sub * 8;
    const bf16_t* vbase = kbase + (size_t)hkv * KV_BLOCK * HD;

    float m_run = -INFINITY, l_run = 0.f, acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    for (int kb = wb; kb < we; kb += KW) {
        uint4 kr[NL], vr[NL];
#pragma unroll
        for (int t = 0; t < NL; ++t) {
            const int key = min(kb + t * KPL + kq, we - 1);
            const size_t off = (size_t)s_bt[(key >> 4) - b0] * blk_elems + (size_t)(key & 15) * HD;
            kr[t] = ld_stream16(kbase + off);
            vr[t] = ld_stream16(vbase + off);
        }
        float sc[NL];
        float mr = -INFINITY;
#pragma unroll
        for (int t = 0; t < NL; ++t) {
            float kv[8];
            load8<bf16_t>(reinterpret_cast<const bf16_t*>(&kr[t]), kv);
            float dot = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) dot = fmaf(q[j], kv[j], dot);
            dot = LPK == 8 ? sum_lanes8(dot) : sum_lanes16(dot);
            sc[t] = (kb + t * KPL + kq < we) ? dot * scale_log2 : -INFINITY;
            mr = fmaxf(mr, sc[t]);
        }
        mr = wave_max(mr);
        const float m_new = fmaxf(m_run, mr);
        const float alpha = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] *= alpha;
#pragma unroll
        for (int t = 0; t < NL; ++t) {
            const float p = (sc[t] == -INFINITY) ? 0.f : fast_exp2(sc[t] - m_new);
            l_run += p;
            float vv[8];
            load8<bf16_t>(reinterpret_cast<const bf16_t*>(&vr[t]), vv);
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[j] = fmaf(p, vv[j], acc[j]);
        }
        m_run = m_new;
    }
    // lanes of one key slot hold the same l; sum over the key slots
    auto slots_sum = [&](float v) {
        if (LPK == 8) v += dpp_f<DPP_ROR8>(v);
        v += swz_xor16_f(v);
        return v + __shfl_xor(v, 32, 64);
    };
    l_run = slots_sum(l_run);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = slots_sum(acc[j]);
    if (kq == 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) s_o[wave][sub * 8 + j] = acc[j];
    }
    if (lane == 0) { s_ml[wave][0] = m_run; s_ml[wave][1] = l_run; }
    __syncthreads();
    // the chunk's state: the four waves merged in wave order
    float M = -INFINITY, L = 0.f, o = 0.f;
    if (tid < HD) {
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, s_ml[w][0]);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float wt = (s_ml[w][0] == -INFINITY) ? 0.f : fast_exp2(s_ml[w][0] - M);
            L += wt * s_ml[w][1];
            o += wt * s_o[w][tid];
        }
    }
    bf16_t* const out = (bf16_t*)a.O + (size_t)i * a.ldo + h * HD;
    if (nch == 1) {
        if (tid < HD) st_elem<bf16_t>(out + tid, kvlen > 0 ? o / L : 0.f);
        return;
    }
    // several chunks: store this chunk's state, the last workgroup merges
    const int sh = i * a.q_heads + h;
    const __amdgpu_buffer_rsrc_t part = coherent_rsrc(a.part + (size_t)sh * a.max_splits * (HD + 2));
    if (tid < HD) st_coherent1(part, (c * (HD + 2) + tid) * 4, o);
    if (tid == 0) {
        st_coherent1(part, (c * (HD + 2) + HD) * 4, M);
        st_coherent1(part, (c * (HD + 2) + HD + 1) * 4, L);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0)
        s_last = __hip_atomic_fetch_add(a.counters + sh, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                 (unsigned)(nch - 1);
    __syncthreads();
    if (!s_last) return;
    if (tid < HD) {
        float Mt = -INFINITY;
        for (int k = 0; k < nch; ++k) Mt = fmaxf(Mt, ld_coherent1(part, (k * (HD + 2) + HD) * 4));
        float Lt = 0.f, ot = 0.f;
        for (int k = 0; k < nch; ++k) {
            const float mk = ld_coherent1(part, (k * (HD + 2) + HD) * 4);
            const float wt = (mk == -INFINITY) ? 0.f : fast_exp2(mk - Mt);
            Lt += wt * ld_coherent1(part, (k * (HD + 2) + HD + 1) * 4);
            ot += wt * ld_coherent1(part, (k * (HD + 2) + tid) * 4);
        }
        st_elem<bf16_t>(out + tid, ot / Lt);
    }
    if (tid == 0) __hip_atomic_store(a.counters + sh, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// grid (n, q_heads), HD threads
template <typename T, int HD>
__global__ void attn_decode_combine_kernel(AttnDecodeArgs a)
{
    const int i = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
    const int nsp = (a.kv_len[i] + ATTN_DEC_CHUNK - 1) / ATTN_DEC_CHUNK;
    const float* part = a.part + ((size_t)i * a.q_heads + h) * a.max_splits * (HD + 2);
    float M = -INFINITY;
    for (int s = 0; s < nsp; ++s) M = fmaxf(M, part[s * (HD + 2) + HD]);
    float L = 0.f, o = 0.f;
    for (int s = 0; s < nsp; ++s) {
        const float w = fast_exp2(part[s * (HD + 2) + HD] - M);
        L += w * part[s * (HD + 2) + HD + 1];
        o += w * part[s * (HD + 2) + d];
    }
    st_elem<T>((T*)a.O + (size_t)i * a.ldo + h * HD + d, o / L);
}

void attn_decode(const AttnDecodeArgs& a, hipStream_t s) {
    if (a.n <= 0) return;
    const int hd = a.kv.head_dim;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    dim3 g1(a.n, a.q_heads, a.max_splits), g2(a.n, a.q_heads);
    if (a.bf16) {
        // chunks of the longest sequence the part buffer is laid out for
        const int keys = a.max_splits * ATTN_DEC_CHUNK;
        if (hd == 64) {
            constexpr int CK = attn_decode_chunk<64>();
            hipLaunchKernelGGL(attn_decode_bf16_kernel<64>, dim3(a.n, a.q_heads, (keys + CK - 1) / CK), dim3(256), 0,
                               s, a, scale_log2);
        } else {
            constexpr int CK = attn_decode_chunk<128>();
            hipLaunchKernelGGL(attn_decode_bf16_kernel<128>, dim3(a.n, a.q_heads, (keys + CK - 1) / CK), dim3(256), 0,
                               s, a, scale_log2);
        }
    } else {
        if (hd == 64) {
            hipLaunchKernelGGL((attn_decode_split_kernel<float, 64>), g1, dim3(256), 0, s, a, scale_log2);
            hipLaunchKernelGGL((attn_decode_combine_kernel<float, 64>), g2, dim3(64), 0, s, a);
        } else {
            hipLaunchKernelGGL((attn_decode_split_kernel<float, 128>), g1, dim3(256), 0, s, a, scale_log2);
            hipLaunchKernelGGL((attn_decode_combine_kernel<float, 128>), g2, dim3(128), 0, s, a);
        }
    }
}

}  // namespace ebrl
