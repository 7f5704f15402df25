// Projections y = x W^T of every linear layer (W stored [out, in]).
//
// bf16 path, three kernels, all on v_mfma_f32_16x16x32_bf16 with fp32
// accumulation.  The weight tile feeds the MFMA "A" operand and the
// activation tile the "B" operand, so a lane ends up owning four consecutive
// output columns of one row: a SwiGLU gate/up pair lands in the same lane
// (weights packed in 32-row groups: 16 gate rows, then the 16 matching up
// rows), and so does a rotary pair of the fused QKV projection.
//  * gemm_bf16_big_kernel (M >= 256: prefill, ViT, flow expert): 256 x 256,
//    192 x 256 or 128 x 128 tiles (16, 12 or 8 waves), operands DMA'd
//    global -> LDS, epilogue staged through LDS for whole-row stores.
//  * gemm_bf16_decode_kernel (decode, M <= 256): 32-, 64- or 96-column slices, per-wave
//    LDS pipelines fed by whole-line DMA; K split across workgroups only for
//    narrow outputs, the partials summed in split order inside the kernel by
//    the last workgroup of each tile.
//  * gemm_bf16_kernel: register-staged LDS tiles for the remaining shapes
//    (K not a multiple of 64), with split-K partials reduced in split order
//    by splitk_reduce_kernel.
// fp32 path (fp32 policies): LDS-tiled FMA kernel with the same epilogues.
// Every choice that orders a sum -- the K split count -- is a function of
// (N, K) alone (plus M >= 256 for the large-M kernel); tile shapes, slice
// widths and block order, which may follow M and the stream's CU count,
// never change an element's summation order.  Results therefore do not
// depend on timing, on the number of compute units or on how many rows a
// decode call holds.
#include <type_traits>

#include "kernels.h"

namespace ebrl {

// ------------------------------------------------------------ epilogues --

struct EpiF32 {
    float* C; int ldc;
    EBRL_DEV void operator()(int m, int n, float a, float b, float c, float d) const {
        st4<float>(C + (size_t)m * ldc + n, a, b, c, d);
    }
};
template <typename T> struct EpiStore {
    T* C; int ldc;
    EBRL_DEV void operator()(int m, int n, float a, float b, float c, float d) const {
        st4<T>(C + (size_t)m * ldc + n, a, b, c, d);
    }
};
// Residual add; with xb set it also stores the updated rows in bf16 (the
// operand of a following projection that folds in the RMSNorm).
struct EpiResid {
    float* C; int ldc; bf16_t* xb; int ldxb;
    EBRL_DEV void operator()(int m, int n, float a, float b, float c, float d) const {
        float4* p = reinterpret_cast<float4*>(C + (size_t)m * ldc + n);
        float4 r = *p;
        r.x += a; r.y += b; r.z += c; r.w += d;
        *p = r;
        if (xb) st4<bf16_t>(xb + (size_t)m * ldxb + n, r.x, r.y, r.z, r.w);
    }
};
// Output row m goes to row_base[m / group] + m % group; optionally adds a
// per-(m % group) row of `add` (position embedding).
template <typename TA> struct EpiRemap {
    float* C; int ldc; const int* row_base; int group; const TA* add; int add_ld;
    EBRL_DEV void operator()(int m, int n, float a, float b, float c, float d) const {
        int g = m / group, r = m - g * group;
        size_t dst = (size_t)(row_base ? row_base[g] + r : m);
        if (add) {
            const TA* ap = add + (size_t)r * add_ld + n;
            a += ld_elem<TA>(ap); b += ld_elem<TA>(ap + 1);
            c += ld_elem<TA>(ap + 2); d += ld_elem<TA>(ap + 3);
        }
        st4<float>(C + dst * ldc + n, a, b, c, d);
    }
};
EBRL_DEV float silu_f(float g) { return g / (1.0f + __expf(-g)); }
// Paired epilogue: gate at packed column n (n % 32 < 16), up at n + 16.
template <typename T> struct EpiSwiGLU {
    T* H; int ldh;
    EBRL_DEV void pair(int m, int n, const float* g, const float* u) const {
        int col = (n >> 5) * 16 + (n & 15);
        st4<T>(H + (size_t)m * ldh + col, silu_f(g[0]) * u[0], silu_f(g[1]) * u[1],
               silu_f(g[2]) * u[2], silu_f(g[3]) * u[3]);
    }
};

// Paired epilogue of the fused QKV projection: columns n (first half of a
// head-local 32-row group) and n + 16 hold rotation partners e and e + hd/2.
template <typename T> struct EpiQKV {
    T* Q; int ldq; T* kv; const int* bt; int bt_stride; int hq, hkv, hd;
    const int* seq_env; const int* row_seq; const int* row_pos;
    const float* cos_tab; const float* sin_tab; int use_rope;
    // Per-row part of the destination: the row's position and the element
    // offset of its token row in head 0's K block (paged cache).
    EBRL_DEV int4 row_info(int m) const {
        const int pos = row_pos[m];
        const int env = seq_env[row_seq[m]];
        const int blk = bt[(size_t)env * bt_stride + (pos >> 4)];
        const size_t off = (size_t)blk * 2 * hkv * KV_BLOCK * hd + (size_t)(pos & 15) * hd;
        return make_int4(pos, (int)(uint32_t)off, (int)(uint32_t)(off >> 32), 0);
    }
    EBRL_DEV void pair_at(int4 ri, int m, int n, const float* x1, const float* x2) const {
        const int qn = hq * hd, kn = hkv * hd;
        const int region = n < qn ? 0 : (n < qn + kn ? 1 : 2);
        const int local = n - (region == 0 ? 0 : (region == 1 ? qn : qn + kn));
        const int h = local / hd, pc = local - h * hd;
        const int e = (pc >> 5) * 16 + (pc & 15);
        const int half = hd >> 1;
        const int pos = ri.x;
        float a[4], b[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) { a[t] = x1[t]; b[t] = x2[t]; }
        if (region < 2 && use_rope) {
            const float4 c = *reinterpret_cast<const float4*>(cos_tab + (size_t)pos * half + e);
            const float4 sn = *reinterpret_cast<const float4*>(sin_tab + (size_t)pos * half + e);
            const float cc[4] = {c.x, c.y, c.z, c.w}, ss[4] = {sn.x, sn.y, sn.z, sn.w};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                a[t] = x1[t] * cc[t] - x2[t] * ss[t];
                b[t] = x2[t] * cc[t] + x1[t] * ss[t];
            }
        }
        T* dst;
        if (region == 0) {
            dst = Q + (size_t)m * ldq + h * hd;
        } else {
            const size_t off = (size_t)(uint32_t)ri.y | ((size_t)(uint32_t)ri.z << 32);
            dst = kv + off + ((size_t)(region == 2 ? hkv : 0) + h) * KV_BLOCK * hd;
        }
        st4<T>(dst + e, a[0], a[1], a[2], a[3]);
        st4<T>(dst + e + half, b[0], b[1], b[2], b[3]);
    }
    EBRL_DEV void pair(int m, int n, const float* x1, const float* x2) const {
        pair_at(row_info(m), m, n, x1, x2);
    }
};
// Epilogues whose per-row work the large-M kernel hoists out of the column loop.
template <class E> struct epi_row_info : std::false_type {};
template <typename T> struct epi_row_info<EpiQKV<T>> : std::true_type {};
template <typename T> EpiQKV<T> make_epi_qkv(const RopeKVArgs& r) {
    return EpiQKV<T>{(T*)r.Q, r.ldq, (T*)r.kv.base, r.kv.block_table, r.kv.bt_stride, r.q_heads,
                     r.kv.kv_heads, r.kv.head_dim, r.seq_env, r.row_seq, r.row_pos, r.cos_tab, r.sin_tab,
                     (int)r.use_rope};
}

// ------------------------------------------------------- bf16 MFMA GEMM --

constexpr int BK = 64;
constexpr int LDSW = BK + 8;  // padded LDS row (bf16 elements)

template <int BM, int BN, int WM, int WN, bool PAIRED, bool SPLIT, class Epi>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(
    const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb, int M, int N,
    int K, int k_per_split, float* __restrict__ ws, Epi epi)
{
    static_assert(WM * WN == 4, "4 waves");
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 16, TN = WTN / 16;
    static_assert(TM >= 1 && TN >= 1, "wave tile");
    static_assert(!PAIRED || (TN % 2 == 0), "paired epilogue needs tile pairs");
    constexpr int A_CHUNKS = BM * (BK / 8), B_CHUNKS = BN * (BK / 8);
    constexpr int A_ITERS = (A_CHUNKS + 255) / 256, B_ITERS = (B_CHUNKS + 255) / 256;

    __shared__ __attribute__((aligned(16))) bf16_t sA[2][BM * LDSW];
    __shared__ __attribute__((aligned(16))) bf16_t sB[2][BN * LDSW];

    const int tid = threadIdx.x;
    const int tiles_n = (N + BN - 1) / BN;
    const int tm_idx = blockIdx.x / tiles_n, tn_idx = blockIdx.x - tm_idx * tiles_n;
    const int m0 = tm_idx * BM, n0 = tn_idx * BN;
    const int k_begin = blockIdx.y * k_per_split;
    const int k_end = min(K, k_begin + k_per_split);
    const int nk = (k_end - k_begin + BK - 1) / BK;

    uint4 ra[A_ITERS], rb[B_ITERS];
    auto load_tiles = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_ITERS; ++i) {
            int c = tid + 256 * i;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (c < A_CHUNKS) {
                int row = c >> 3, kc = (c & 7) * 8;
                int gr = min(m0 + row, M - 1), gk = k0 + kc;
                if (gk < k_end) v = *reinterpret_cast<const uint4*>(A + (size_t)gr * lda + gk);
            }
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < B_ITERS; ++i) {
            int c = tid + 256 * i;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (c < B_CHUNKS) {
                int row = c >> 3, kc = (c & 7) * 8;
                int gr = min(n0 + row, N - 1), gk = k0 + kc;
                if (gk < k_end) v = *reinterpret_cast<const uint4*>(B + (size_t)gr * ldb + gk);
            }
            rb[i] = v;
        }
    };
    auto store_tiles = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_ITERS; ++i) {
            int c = tid + 256 * i;
            if (c < A_CHUNKS) {
                int row = c >> 3, kc = (c & 7) * 8;
                *reinterpret_cast<uint4*>(&sA[buf][row * LDSW + kc]) = ra[i];
            }
        }
#pragma unroll
        for (int i = 0; i < B_ITERS; ++i) {
            int c = tid + 256 * i;
            if (c < B_CHUNKS) {
                int row = c >> 3, kc = (c & 7) * 8;
                *reinterpret_cast<uint4*>(&sB[buf][row * LDSW + kc]) = rb[i];
            }
        }
    };

    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave / WN, wn = wave - wm * WN;
    const int r = lane & 15, g = lane >> 4;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    if (nk > 0) {
        load_tiles(k_begin);
        store_tiles(0);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const int buf = kt & 1;
            if (kt + 1 < nk) load_tiles(k_begin + (kt + 1) * BK);
#pragma unroll
            for (int ks = 0; ks < BK / 32; ++ks) {
                bf16x8 wa[TN], xb[TM];
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    wa[j] = *reinterpret_cast<const bf16x8*>(
                        &sB[buf][(wn * WTN + j * 16 + r) * LDSW + ks * 32 + g * 8]);
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    xb[i] = *reinterpret_cast<const bf16x8*>(
                        &sA[buf][(wm * WTM + i * 16 + r) * LDSW + ks * 32 + g * 8]);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[j], xb[i], acc[i][j],
                                                                            0, 0, 0);
            }
            if (kt + 1 < nk) store_tiles(buf ^ 1);
            __syncthreads();
        }
    }

    // lane owns rows m = ... + r, columns n = ... + 4g .. 4g+3 of each tile
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int m = m0 + wm * WTM + i * 16 + r;
        if (m >= M) continue;
        if constexpr (SPLIT) {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = n0 + wn * WTN + j * 16 + 4 * g;
                if (n < N)
                    st4<float>(ws + ((size_t)blockIdx.y * M + m) * N + n, acc[i][j][0],
                               acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
        } else if constexpr (PAIRED) {
#pragma unroll
            for (int j = 0; j < TN; j += 2) {
                const int n = n0 + wn * WTN + j * 16 + 4 * g;
                if (n < N) {
                    float gv[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
                    float uv[4] = {acc[i][j + 1][0], acc[i][j + 1][1], acc[i][j + 1][2],
                                   acc[i][j + 1][3]};
                    epi.pair(m, n, gv, uv);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = n0 + wn * WTN + j * 16 + 4 * g;
                if (n < N) epi(m, n, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
        }
    }
}


// ------------------------------------------------ bf16 MFMA GEMM, large M --
// 256 x 256 macro tiles, 16 waves in 4 x 4 (64 x 64 per wave, four waves
// per SIMD so that one wave's LDS waits overlap another's MFMAs); the
// 192 x 256 and 128 x 128 variants run 12 waves of 64 x 64 and 8 of 64 x 32.
// Operands go global -> LDS with global_load_lds_dwordx4 (no VGPR staging):
// a wave instruction writes 64 lanes x 16 bytes contiguously, so the tile is
// stored as 16-byte chunks, chunk (row, c) of a 64-element row at position
// row * 8 + (c ^ (row & 7)); the XOR makes the MFMA fragment reads of 8
// consecutive rows hit 8 different bank groups.  Two LDS stages: the loads of
// K tile t+1 are in flight while tile t is multiplied.  Block ids are
// remapped so that consecutive tiles of one row band run on the same XCD
// (the dispatcher deals block ids round-robin over the 8 XCDs).
typedef __attribute__((address_space(3))) void* lds_ptr_t;

EBRL_DEV void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0); }

// s_waitcnt on the vector-memory counter only (gfx9 encoding: expcnt and
// lgkmcnt fields at their maxima).
template <int N> EBRL_DEV void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | 0xF00 | ((N >> 4) << 14));
}

// global_load_lds_dwordx4 issued as inline assembly: the compiler neither
// counts these loads nor guards LDS reads against them, so its own waits
// stay partial; kernels that use it wait on vmcnt and synchronise
// themselves before reading what the DMA filled.
EBRL_DEV void dma16_to_lds(const void* g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(g), "s"(lds_addr) : "memory", "m0");
}
// The same with the non-temporal hint, for weights that no other workgroup of
// the launch reads again (streaming them keeps the activations cached).
EBRL_DEV void dma16_to_lds_nt(const void* g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                 :: "v"(g), "s"(lds_addr) : "memory", "m0");
}


// The same DMA in its scalar-base form: a wave-uniform 64-bit base in SGPRs
// plus a 32-bit per-lane byte offset, so a wave's row offsets stay fixed
// across K tiles (only the scalar base advances) and take one VGPR each.
EBRL_DEV void dma16_to_lds_s(const void* sbase, uint32_t voff, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(voff), "s"(sbase), "s"(lds_addr) : "memory", "m0");
}

// ROWS x 64 bf16 of G (rows row0_g.., columns k0..k0+63; rows past
// rows_valid repeat the last valid row) into lds_tile, 16-byte chunk c of
// row r at position r * 8 + (c ^ (r & 7)).  The loads go through inline
// assembly: callers wait on vmcnt and synchronise before reading the tile.
template <int ROWS, int NW>
EBRL_DEV void load_tile_lds(const bf16_t* __restrict__ G, int ld, int row0_g, int rows_valid, int k0,
                            bf16_t* lds_tile, int wave, int lane) {
    // base and LDS addresses are wave-uniform: pinned to SGPRs (readfirstlane
    // returns int: each half goes through uint32_t, so the low half is
    // zero-extended)
    const uint64_t b = (uint64_t)(uintptr_t)(G + (size_t)row0_g * ld + k0);
    const uint32_t b_hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32));
    const uint32_t b_lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
    const void* const base = (const void*)(uintptr_t)(((uint64_t)b_hi << 32) | (uint64_t)b_lo);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)lds_tile;
    const int last = rows_valid - 1 - row0_g;
    auto group = [&](int r0) {   // rows r0 .. r0+7, one instruction
        const int row = r0 + (lane >> 3);
        const int c = (lane & 7) ^ (row & 7);
        const uint32_t voff = (uint32_t)(min(row, last) * ld + c * 8) * 2u;
        dma16_to_lds_s(base, voff, __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)r0 * 128u));
    };
    if constexpr (ROWS % (8 * NW) == 0) {
        // each of the NW waves fills ROWS/NW consecutive rows
#pragma unroll
        for (int j = 0; j < ROWS / (8 * NW); ++j) group(wave * (ROWS / NW) + j * 8);
    } else {
        // 8-row groups dealt round-robin over the waves
#pragma unroll
        for (int j = 0; j < (ROWS / 8 + NW - 1) / NW; ++j) {
            const int gi = wave + j * NW;
            if (gi < ROWS / 8) group(gi * 8);
        }
    }
}

EBRL_DEV bf16x8 lds_frag(const bf16_t* tile, int row, int c) {
    return *reinterpret_cast<const bf16x8*>(tile + row * 64 + ((c ^ (row & 7)) << 3));
}

// XO: the K loop overlaps the per-tile barrier with MFMAs (below).
template <int BM, int BN, int WM, int WN, bool PAIRED, bool XO, class Epi>
__global__ __launch_bounds__(64 * WM * WN, WM * WN == 8 ? 4 : 1) void gemm_bf16_big_kernel(
    const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb, int M, int N, int K,
    int k_per_split, float* __restrict__ ws, Epi epi)
{
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 16, TN = WTN / 16;
    static_assert(!PAIRED || (TN % 2 == 0), "paired epilogue needs tile pairs");
    // one __shared__ object per stage and operand (the DMA that fills them
    // is inline assembly the compiler does not track: every read of a stage
    // follows an explicit vmcnt wait and a barrier)
    __shared__ __attribute__((aligned(1024))) bf16_t sA0[BM * 64];
    __shared__ __attribute__((aligned(1024))) bf16_t sA1[BM * 64];
    __shared__ __attribute__((aligned(1024))) bf16_t sB0[BN * 64];
    __shared__ __attribute__((aligned(1024))) bf16_t sB1[BN * 64];

    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int bid = blockIdx.x;
    const int nb = gridDim.x;
    if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
    constexpr int G = 4;  // row tiles per group
    const int group = G * tiles_n;
    const int first_m = (bid / group) * G;
    const int gsz = min(tiles_m - first_m, G);
    const int within = bid - (bid / group) * group;
    const int tm_idx = first_m + within % gsz, tn_idx = within / gsz;
    const int m0 = tm_idx * BM, n0 = tn_idx * BN;

    const int k_begin = blockIdx.y * k_per_split;
    const int k_end = min(K, k_begin + k_per_split);
    const int nk = (k_end - k_begin) / 64;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave - (wave / WN) * WN;
    const int r = lane & 15, g = lane >> 4;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Each 64-wide K tile is multiplied as two 32-wide halves.  With XO the
    // barrier that publishes tile t + 1 sits between tile t's halves: before it a
    // wave reads tile t's second-half fragments and multiplies its first
    // half; after it, it issues the DMA of tile t + 2 into the stage tile t
    // has left, multiplies tile t's second half -- operands already in
    // registers, so the MFMA pipes start right after the barrier -- and
    // then reads tile t + 1's first-half fragments behind those MFMAs.
    // Every accumulator still takes its K steps in order, so the bits do
    // not depend on XO.  The 16-wave tile has no registers for the second
    // fragment set (it spills); on 12 waves the overlap measured up to 7 %
    // faster from K 2048 on (one shape 2.5 % slower) and 3 % slower at
    // K 1024, on 8 waves 2-6 % faster at every K.
    static_assert(!XO || WM * WN != 16, "the 16-wave tile runs without the overlap");
    bf16x8 w0[TN], x0[TM], w1[TN], x1[TM];
    auto read_half = [&](const bf16_t* ta, const bf16_t* tb, int ks, bf16x8 (&w)[TN], bf16x8 (&x)[TM]) {
#pragma unroll
        for (int j = 0; j < TN; ++j) w[j] = lds_frag(tb, wn * WTN + j * 16 + r, ks * 4 + g);
#pragma unroll
        for (int i = 0; i < TM; ++i) x[i] = lds_frag(ta, wm * WTM + i * 16 + r, ks * 4 + g);
    };
    auto mma = [&](const bf16x8 (&w)[TN], const bf16x8 (&x)[TM]) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[j], x[i], acc[i][j], 0, 0, 0);
    };
    // tile t is in stage (ta, tb), tile t + 1 in (na, nb_); tile t + 2 goes
    // into (ta, tb)
    auto step = [&](int t, bf16_t* ta, bf16_t* tb, const bf16_t* na, const bf16_t* nb_) {
        read_half(ta, tb, 1, w1, x1);
        mma(w0, x0);
        __builtin_amdgcn_sched_barrier(0);
        // own fragment reads of this stage done, own DMA of tile t + 1 landed
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        if (t + 2 < nk) {
            load_tile_lds<BM, NW>(A, lda, m0, M, k_begin + (t + 2) * 64, ta, wave, lane);
            load_tile_lds<BN, NW>(B, ldb, n0, N, k_begin + (t + 2) * 64, tb, wave, lane);
        }
        mma(w1, x1);
        __builtin_amdgcn_sched_barrier(0);
        if (t + 1 < nk) read_half(na, nb_, 0, w0, x0);
    };

    // Without the overlap: a whole K tile's fragments are read, multiplied,
    // then the wave waits at the barrier.
    auto compute = [&](const bf16_t* ta, const bf16_t* tb) {
        read_half(ta, tb, 0, w0, x0);
        read_half(ta, tb, 1, w1, x1);
        mma(w0, x0);
        mma(w1, x1);
    };

    if (nk > 0) {
        load_tile_lds<BM, NW>(A, lda, m0, M, k_begin, sA0, wave, lane);
        load_tile_lds<BN, NW>(B, ldb, n0, N, k_begin, sB0, wave, lane);
        wait_vm_all();
        __syncthreads();
        if constexpr (!XO) {
            for (int kt = 0; kt < nk; kt += 2) {
                if (kt + 1 < nk) {
                    load_tile_lds<BM, NW>(A, lda, m0, M, k_begin + (kt + 1) * 64, sA1, wave, lane);
                    load_tile_lds<BN, NW>(B, ldb, n0, N, k_begin + (kt + 1) * 64, sB1, wave, lane);
                }
                compute(sA0, sB0);
                wait_vm_all();
                __syncthreads();
                if (kt + 1 < nk) {
                    if (kt + 2 < nk) {
                        load_tile_lds<BM, NW>(A, lda, m0, M, k_begin + (kt + 2) * 64, sA0, wave, lane);
                        load_tile_lds<BN, NW>(B, ldb, n0, N, k_begin + (kt + 2) * 64, sB0, wave, lane);
                    }
                    compute(sA1, sB1);
                    wait_vm_all();
                    __syncthreads();
                }
            }
        } else {
            if (nk > 1) {
                load_tile_lds<BM, NW>(A, lda, m0, M, k_begin + 64, sA1, wave, lane);
                load_tile_lds<BN, NW>(B, ldb, n0, N, k_begin + 64, sB1, wave, lane);
            }
            read_half(sA0, sB0, 0, w0, x0);
            for (int kt = 0; kt < nk; kt += 2) {
                step(kt, sA0, sB0, sA1, sB1);
                if (kt + 1 < nk) step(kt + 1, sA1, sB1, sA0, sB0);
            }
        }
    }

    // Epilogue through LDS (free once every wave has passed the loop's last
    // barrier): a wave stages 16 rows x 64 columns of its tile at a time and
    // reads them back row-contiguous, so that each store (and the residual
    // read) covers 256-byte fp32 / 64-128-byte bf16 row segments instead of
    // 16-32-byte pieces of 16 rows.  Rows are padded to 68 floats so the
    // fragment-layout writes spread over the banks.
    static_assert(WTN == 64 || WTN == 32, "staging assumes 64- or 32-column wave tiles");
    constexpr int SROW = WTN + 4;
    constexpr int PER_A = (BM * 64 * 2) / (16 * SROW * 4), PER_B = (BN * 64 * 2) / (16 * SROW * 4);
    static_assert(2 * (PER_A + PER_B) >= NW, "staging space");
    static_assert(WTM == 64, "one row per lane in the per-row epilogue data");
    // per-row epilogue data of the wave's 64 rows, one row per lane
    __shared__ int4 s_row[epi_row_info<Epi>::value ? NW : 1][64];
    if constexpr (epi_row_info<Epi>::value)
        s_row[wave][lane] = epi.row_info(min(m0 + wm * WTM + lane, M - 1));
    bf16_t* const region = wave < PER_A ? sA0 : (wave < 2 * PER_A ? sA1 : (wave < 2 * PER_A + PER_B ? sB0 : sB1));
    const int slot = wave < PER_A ? wave : (wave < 2 * PER_A ? wave - PER_A
                                            : (wave < 2 * PER_A + PER_B ? wave - 2 * PER_A : wave - 2 * PER_A - PER_B));
    float* const stage = reinterpret_cast<float*>(region) + slot * 16 * SROW;
    const int ncol0 = n0 + wn * WTN;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
            *reinterpret_cast<f32x4*>(stage + r * SROW + j * 16 + 4 * g) = acc[i][j];
        const int mrow0 = m0 + wm * WTM + i * 16;
        if constexpr (PAIRED) {
            // WTN / 8 lanes per row: gate columns c (c % 32 < 16) with up partner c + 16
            constexpr int LPR = WTN / 8;
#pragma unroll
            for (int pass = 0; pass < LPR / 4; ++pass) {
                const int row = pass * (64 / LPR) + lane / LPR;
                const int c = ((lane % LPR) >> 2) * 32 + (lane & 3) * 4;
                const f32x4 gv4 = *reinterpret_cast<const f32x4*>(stage + row * SROW + c);
                const f32x4 uv4 = *reinterpret_cast<const f32x4*>(stage + row * SROW + c + 16);
                const int m = mrow0 + row, n = ncol0 + c;
                if (m < M && n < N) {
                    float gv[4] = {gv4[0], gv4[1], gv4[2], gv4[3]};
                    float uv[4] = {uv4[0], uv4[1], uv4[2], uv4[3]};
                    if constexpr (epi_row_info<Epi>::value) epi.pair_at(s_row[wave][i * 16 + row], m, n, gv, uv);
                    else epi.pair(m, n, gv, uv);
                }
            }
        } else {
            // WTN / 4 lanes per row, four columns each
            constexpr int LPR = WTN / 4;
#pragma unroll
            for (int pass = 0; pass < LPR / 4; ++pass) {
                const int row = pass * (64 / LPR) + lane / LPR;
                const int c = (lane % LPR) * 4;
                const f32x4 v = *reinterpret_cast<const f32x4*>(stage + row * SROW + c);
                const int m = mrow0 + row, n = ncol0 + c;
                if (m < M && n < N) epi(m, n, v[0], v[1], v[2], v[3]);
            }
        }
    }
}


// ------------------------------------------- bf16 GEMM, decode-sized M --
// M <= 256 (one row per environment), K % 64 == 0.  A workgroup owns a
// 32-, 64- or 96-column slice of the output, at most 64 rows (further row tiles in more
// workgroups) and a contiguous range of 64-wide K groups; the range is the
// whole K unless the column slices alone are too few to occupy the chip.  The
// four waves split that range and run independent pipelines: each wave
// streams its weight and activation rows into its own LDS region with
// global_load_lds_dwordx4 (one instruction = 8 rows x 128 contiguous bytes,
// whole cache lines), three buffers deep for 64-column slices where they fit
// the LDS (two otherwise), and multiplies from LDS.  Loading
// whole 128-byte row segments per instruction roughly doubles the rate a CU
// sustains compared with loading 16 rows x 64 bytes straight into MFMA
// register layout.  The waves' tiles are summed in wave order through LDS.
// With several K splits each workgroup stores its partial tile, and the
// workgroup that finishes a tile last (a device-scope counter per tile) sums
// the partials in split order, runs the epilogue and clears the counter for
// the next call.  An element's summation order depends only on (N, K).
constexpr int DEC_BN = 64;   // column slice of the split rule (the kernel also runs 32- and 96-wide slices)
constexpr int DEC_MAX_SPLITS = 16;
constexpr int DEC_TILE_FLOATS = 64 * 64;   // partial-tile stride in the workspace
constexpr int DEC_MAX_COUNTERS = 4096;

// One wave's DMA of ROWS rows x 64 bf16 (K group k0) into `lds`: row q of the
// group sits in instruction q / 8, lane (q % 8) * 8 + (c ^ (q % 8)) holds its
// 16-byte chunk c (the XOR spreads a fragment read over the banks).  Each
// wave reads only the region its own DMA fills.
template <int ROWS, bool NT = false>
EBRL_DEV void dec_dma(const bf16_t* __restrict__ G, int ld, int row0, int rows_valid, int k0, bf16_t* lds,
                      int lane) {
    const int q = lane >> 3, c = (lane & 7) ^ q;
    const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_ptr_t)lds);
#pragma unroll
    for (int t = 0; t < ROWS / 8; ++t) {
        const int gr = min(row0 + t * 8 + q, rows_valid - 1);
        if constexpr (NT) dma16_to_lds_nt(G + (size_t)gr * ld + k0 + c * 8, base + t * 1024);
        else dma16_to_lds(G + (size_t)gr * ld + k0 + c * 8, base + t * 1024);
    }
}
EBRL_DEV bf16x8 dec_frag(const bf16_t* lds, int row, int c) {
    return *reinterpret_cast<const bf16x8*>(lds + (row >> 3) * 512 + ((row & 7) * 8 + (c ^ (row & 7))) * 8);
}

template <int TM, int BN, bool NTW, bool NORM, bool PAIRED, class Epi>
__global__ __launch_bounds__(256) void gemm_bf16_decode_kernel(
    const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ W, int ldw, int M, int N,
    int K, int groups_per_split, int splits, int m_tiles, float* __restrict__ ws,
    unsigned* __restrict__ counters, float norm_eps, Epi epi)
{
    constexpr int TN = BN / 16;
    static_assert(!PAIRED || TN % 2 == 0, "paired epilogue needs fragment pairs");
    constexpr int FR = TM * TN;            // output fragments per wave
    constexpr int WE = BN * 64;            // bf16 per wave per buffer: weights
    constexpr int XE = TM * 16 * 64;       //                             activations
    constexpr int NDMA = (BN + TM * 16) / 8;       // DMA instructions per K group
    // Three buffers per wave (two K groups in flight while a third is
    // multiplied) for 64-column slices where they fit the LDS, else two:
    // measured 1-13 % more bandwidth on the 7B-class decode shapes at 1-32
    // rows; 32-column slices (small weights, launch-latency bound) lost
    // up to 9 % from the larger LDS footprint.
    constexpr int STAGES = (BN == 64 && 3 * 4 * (WE + XE) * 2 <= 150 * 1024) ? 3 : 2;
    // one __shared__ object per buffer and operand, so that the compiler can
    // tell the buffer being read from the one the DMA is filling
    __shared__ __attribute__((aligned(1024))) bf16_t sW0[4 * WE];
    __shared__ __attribute__((aligned(1024))) bf16_t sX0[4 * XE];
    __shared__ __attribute__((aligned(1024))) bf16_t sW1[4 * WE];
    __shared__ __attribute__((aligned(1024))) bf16_t sX1[4 * XE];
    __shared__ __attribute__((aligned(1024))) bf16_t sW2[STAGES == 3 ? 4 * WE : 1];
    __shared__ __attribute__((aligned(1024))) bf16_t sX2[STAGES == 3 ? 4 * XE : 1];
    // After the main loop (every DMA landed, a barrier passed) the staging
    // buffers hold the waves' tiles for the reduction -- wave w's region in
    // sW0, then sX0, then sW1, none straddling two buffers -- and sX1 holds
    // the per-row sums of squares and the last-workgroup flag (96-column
    // slices of 64 rows fill the whole 160 KB with the two stages).
    constexpr int RB = FR * 64 * 16;   // bytes of one wave's tile
    constexpr int CW = (int)sizeof(sW0) / RB, CX = (int)sizeof(sX0) / RB;
    static_assert(CW + CX + CW >= 4, "reduction buffer");
    static_assert((NORM ? 4 * TM * 16 * 4 : 0) + 4 <= (int)sizeof(sX1), "row sums and flag");
    float (*const s_ssq)[TM * 16] = reinterpret_cast<float (*)[TM * 16]>(sX1);
    int* const s_last = reinterpret_cast<int*>(sX1) + 4 * TM * 16;
    // K-split partial tiles are DEC_TILE_FLOATS apart in the workspace: the
    // plan splits K only for kernels whose tile fits that stride.
    constexpr bool SPLITTABLE = FR * 64 * 4 <= DEC_TILE_FLOATS;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int tiles_n = (N + BN - 1) / BN;
    // XCD-aware order: the dispatcher deals workgroup ids round-robin over
    // the 8 XCDs; XCD x takes the x-th contiguous range of units (the first
    // nb % 8 ranges one longer), so the row tiles of one (column slice,
    // split) pair -- which read the same weights -- run on the same XCD.
    int bid = blockIdx.x;
    {
        const int nb = gridDim.x, x = bid & 7;
        bid = x * (nb >> 3) + min(x, nb & 7) + (bid >> 3);
    }
    const int mt = bid % m_tiles;
    const int unit = bid / m_tiles;
    const int split = unit % splits, nt = unit / splits;
    const int m0 = mt * 16 * TM, n0 = nt * BN;
    const int kgroups = K >> 6;
    const int s_begin = split * groups_per_split;
    const int s_end = min(kgroups, s_begin + groups_per_split);
    const int gpw = (groups_per_split + 3) >> 2;
    const int w_begin = min(s_end, s_begin + wave * gpw);
    const int w_end = min(s_end, w_begin + gpw);

    bf16_t* const w0 = sW0 + wave * WE; bf16_t* const x0 = sX0 + wave * XE;
    bf16_t* const w1 = sW1 + wave * WE; bf16_t* const x1 = sX1 + wave * XE;
    bf16_t* const w2 = sW2 + (STAGES == 3 ? wave * WE : 0);
    bf16_t* const x2 = sX2 + (STAGES == 3 ? wave * XE : 0);
    auto dma = [&](int grp, bf16_t* wl, bf16_t* xl) {
        dec_dma<BN, NTW>(W, ldw, n0, N, grp * 64, wl, lane);
        dec_dma<TM * 16>(A, lda, m0, M, grp * 64, xl, lane);
    };

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    // NORM: per-lane sum of squares of the activation elements it reads
    // (row i * 16 + r, chunks g and 4 + g of every K group of the wave)
    float ssq[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) ssq[i] = 0.f;
    // both 32-wide steps of a K group: fragment reads first, then the MFMAs
    auto compute = [&](const bf16_t* wl, const bf16_t* xl) {
        bf16x8 wa[2][TN], xb[2][TM];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
            for (int j = 0; j < TN; ++j) wa[u][j] = dec_frag(wl, j * 16 + r, u * 4 + g);
#pragma unroll
            for (int i = 0; i < TM; ++i) xb[u][i] = dec_frag(xl, i * 16 + r, u * 4 + g);
        }
        if constexpr (NORM) {
            typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const uint4 w4 = __builtin_bit_cast(uint4, xb[u][i]);
                    const unsigned w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const bf16x2_t pr = __builtin_bit_cast(bf16x2_t, w[e]);
                        ssq[i] = __builtin_amdgcn_fdot2_f32_bf16(pr, pr, ssq[i], false);
                    }
                }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[u][j], xb[u][i], acc[i][j], 0, 0, 0);
    };

    if constexpr (STAGES == 3) {
        // group g sits in buffer (g - w_begin) % 3; multiplying it first puts
        // group g + 2 in flight into the buffer group g - 1 has left
        auto step = [&](int gi, const bf16_t* wc, const bf16_t* xc, bf16_t* wn, bf16_t* xn) {
            if (gi + 2 < w_end) {
                dma(gi + 2, wn, xn);
                wait_vmcnt<2 * NDMA>();
            } else if (gi + 1 < w_end) {
                wait_vmcnt<NDMA>();
            } else {
                wait_vmcnt<0>();
            }
            compute(wc, xc);
        };
        if (w_begin < w_end) dma(w_begin, w0, x0);
        if (w_begin + 1 < w_end) dma(w_begin + 1, w1, x1);
        for (int gi = w_begin; gi < w_end; gi += 3) {
            step(gi, w0, x0, w2, x2);
            if (gi + 1 >= w_end) break;
            step(gi + 1, w1, x1, w0, x0);
            if (gi + 2 >= w_end) break;
            step(gi + 2, w2, x2, w1, x1);
        }
    } else if (w_begin < w_end) {
        dma(w_begin, w0, x0);
        for (int gi = w_begin; gi < w_end; gi += 2) {
            if (gi + 1 < w_end) {
                dma(gi + 1, w1, x1);
                wait_vmcnt<NDMA>();
            } else {
                wait_vmcnt<0>();
            }
            compute(w0, x0);
            if (gi + 1 >= w_end) break;
            if (gi + 2 < w_end) {
                dma(gi + 2, w0, x0);
                wait_vmcnt<NDMA>();
            } else {
                wait_vmcnt<0>();
            }
            compute(w1, x1);
        }
    }

    // waves' tiles through LDS (the staging buffers, once every wave is done)
    __syncthreads();
    auto red_region = [&](int w) -> f32x4* {
        if (w < CW) return reinterpret_cast<f32x4*>(sW0) + w * FR * 64;
        if (w < CW + CX) return reinterpret_cast<f32x4*>(sX0) + (w - CW) * FR * 64;
        return reinterpret_cast<f32x4*>(sW1) + (w - CW - CX) * FR * 64;
    };
    f32x4* const red = red_region(wave);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) red[(i * TN + j) * 64 + lane] = acc[i][j];
    if constexpr (NORM) {
        // lanes r, r + 16, r + 32, r + 48 hold row r's four chunk columns
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            float t = ssq[i];
            t += __shfl_xor(t, 16, 64);
            t += __shfl_xor(t, 32, 64);
            if (g == 0) s_ssq[wave][i * 16 + r] = t;
        }
    }
    __syncthreads();
    auto red_at = [&](int w, int e) -> f32x4 { return red_region(w)[e]; };

    // Output units: one fragment lane (or a gate/up fragment pair) each.
    constexpr int G = PAIRED ? 2 : 1;
    constexpr int UNITS = FR / G * 64;
    constexpr int PER = (UNITS + 255) / 256;
    f32x4 v[PER][G];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int u = tid + 256 * q;
        if (u < UNITS) {
            const int f0 = (u >> 6) * G, l = u & 63;
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const int e = (f0 + h) * 64 + l;
                v[q][h] = ((red_at(0, e) + red_at(1, e)) + red_at(2, e)) + red_at(3, e);
            }
        }
    }

    if (SPLITTABLE && splits > 1) {
        // A workgroup waits for its own partial stores to complete before it
        // bumps the counter; the last one reads the partials only after
        // seeing the final count.
        const int tile = nt * m_tiles + mt;
        const __amdgpu_buffer_rsrc_t part =
            coherent_rsrc(ws + (size_t)tile * splits * DEC_TILE_FLOATS);
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int u = tid + 256 * q;
            if (u < UNITS) {
                const int f0 = (u >> 6) * G, l = u & 63;
#pragma unroll
                for (int h = 0; h < G; ++h)
                    st_coherent4(part, (split * DEC_TILE_FLOATS + ((f0 + h) * 64 + l) * 4) * 4, v[q][h]);
            }
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0)
            *s_last = __hip_atomic_fetch_add(counters + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                      (unsigned)(splits - 1);
        __syncthreads();
        if (!*s_last) return;
        // all splits' loads in flight at once, then summed in split order
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int u = tid + 256 * q;
            if (u < UNITS) {
                const int f0 = (u >> 6) * G, l = u & 63;
#pragma unroll
                for (int h = 0; h < G; ++h) {
                    const int off = ((f0 + h) * 64 + l) * 16;
                    f32x4 t[DEC_MAX_SPLITS];
#pragma unroll
                    for (int sp = 0; sp < DEC_MAX_SPLITS; ++sp)
                        t[sp] = ld_coherent4(part, min(sp, splits - 1) * DEC_TILE_FLOATS * 4 + off);
                    f32x4 acc_t = t[0];
#pragma unroll
                    for (int sp = 1; sp < DEC_MAX_SPLITS; ++sp)
                        if (sp < splits) acc_t += t[sp];
                    v[q][h] = acc_t;
                }
            }
        }
        if (tid == 0) __hip_atomic_store(counters + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int u = tid + 256 * q;
        if (u < UNITS) {
            const int fg = u >> 6, l = u & 63;
            const int f0 = fg * G;
            const int i = f0 / TN, j = f0 - i * TN;
            const int m = m0 + i * 16 + (l & 15);
            const int n = n0 + j * 16 + 4 * (l >> 4);
            if constexpr (NORM) {
                // RMSNorm of the row, summed over the waves' K ranges in wave order
                const int row = i * 16 + (l & 15);
                const float ss = ((s_ssq[0][row] + s_ssq[1][row]) + s_ssq[2][row]) + s_ssq[3][row];
                const float rs = 1.0f / sqrtf(ss / (float)K + norm_eps);
#pragma unroll
                for (int h = 0; h < G; ++h) v[q][h] *= rs;
            }
            if (m < M && n < N) {
                if constexpr (PAIRED) {
                    float gv[4] = {v[q][0][0], v[q][0][1], v[q][0][2], v[q][0][3]};
                    float uv[4] = {v[q][1][0], v[q][1][1], v[q][1][2], v[q][1][3]};
                    epi.pair(m, n, gv, uv);
                } else {
                    epi(m, n, v[q][0][0], v[q][0][1], v[q][0][2], v[q][0][3]);
                }
            }
        }
    }
}


// ------------------------------------------------------------ fp32 GEMM --
// 64 x 64 tile, BK 16, 256 threads; thread (ty, tx) owns rows 2ty, 2ty+1 and
// columns grp*32 + q*4 + {0..3} and the same +16 (tx = grp*4 + q), so that a
// SwiGLU gate/up pair is in one thread.
template <bool PAIRED, bool SPLIT, class Epi>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int lda,
                                                       const float* __restrict__ B, int ldb, int M,
                                                       int N, int K, int k_per_split,
                                                       float* __restrict__ ws, Epi epi)
{
    constexpr int TBM = 64, TBN = 64, TBK = 16;
    __shared__ float sA[TBK][TBM + 4];
    __shared__ float sB[TBK][TBN + 4];
    const int tid = threadIdx.x;
    const int tiles_n = (N + TBN - 1) / TBN;
    const int tmi = blockIdx.x / tiles_n, tni = blockIdx.x - tmi * tiles_n;
    const int m0 = tmi * TBM, n0 = tni * TBN;
    const int k_begin = blockIdx.y * k_per_split;
    const int k_end = min(K, k_begin + k_per_split);
    const int ty = tid >> 3, tx = tid & 7;
    const int grp = tx >> 2, q = tx & 3;
    int cols[8];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        cols[c] = grp * 32 + q * 4 + c;
        cols[4 + c] = grp * 32 + 16 + q * 4 + c;
    }
    float acc[2][8];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[i][c] = 0.f;

    for (int k0 = k_begin; k0 < k_end; k0 += TBK) {
        // 64 x 16 elements of A and of B: 4 per thread each
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int e = tid + 256 * i;
            int row = e >> 4, kk = e & 15;
            int gk = k0 + kk;
            float va = 0.f, vb = 0.f;
            if (gk < k_end) {
                va = A[(size_t)min(m0 + row, M - 1) * lda + gk];
                vb = B[(size_t)min(n0 + row, N - 1) * ldb + gk];
            }
            sA[kk][row] = va;
            sB[kk][row] = vb;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TBK; ++kk) {
            float a0 = sA[kk][2 * ty], a1 = sA[kk][2 * ty + 1];
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float b = sB[kk][cols[c]];
                acc[0][c] = fmaf(a0, b, acc[0][c]);
                acc[1][c] = fmaf(a1, b, acc[1][c]);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int m = m0 + 2 * ty + i;
        if (m >= M) continue;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int n = n0 + cols[4 * h];
            if (n >= N) continue;
            float* v = &acc[i][4 * h];
            if constexpr (SPLIT) {
                st4<float>(ws + ((size_t)blockIdx.y * M + m) * N + n, v[0], v[1], v[2], v[3]);
            } else if constexpr (PAIRED) {
                if (h == 0) epi.pair(m, n, &acc[i][0], &acc[i][4]);
            } else {
                epi(m, n, v[0], v[1], v[2], v[3]);
            }
        }
    }
}

// Sum split partials in split order, then apply the epilogue.  One thread
// per (row, 4 output columns); for paired epilogues the output columns are
// the gate columns (packed n % 32 < 16).
template <bool PAIRED, class Epi>
__global__ void splitk_reduce_kernel(const float* __restrict__ ws, int splits, int M, int N,
                                     Epi epi)
{
    const int groups = PAIRED ? N / 8 : N / 4;
    const long total = (long)M * groups;
    for (long idx = blockIdx.x * (long)blockDim.x + threadIdx.x; idx < total;
         idx += (long)gridDim.x * blockDim.x) {
        const int m = (int)(idx / groups);
        const int gq = (int)(idx - (long)m * groups);
        int n;
        if (PAIRED) n = (gq >> 2) * 32 + (gq & 3) * 4;
        else n = gq * 4;
        float v[4] = {0.f, 0.f, 0.f, 0.f}, u[4] = {0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < splits; ++s) {
            const float4 a = *reinterpret_cast<const float4*>(ws + ((size_t)s * M + m) * N + n);
            v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w;
            if (PAIRED) {
                const float4 b =
                    *reinterpret_cast<const float4*>(ws + ((size_t)s * M + m) * N + n + 16);
                u[0] += b.x; u[1] += b.y; u[2] += b.z; u[3] += b.w;
            }
        }
        if constexpr (PAIRED) epi.pair(m, n, v, u);
        else epi(m, n, v[0], v[1], v[2], v[3]);
    }
}

// ------------------------------------------------------------- dispatch --

// Tile and split choice depend only on (M, N, K) and the stream's CU count;
// the split count, the only one that orders sums, on (N, K) alone.
struct GemmPlan {
    int bm; int bn; int splits; int k_per_split; bool big;
    bool dec; int steps_per_split; int tm; int m_tiles; int dbn;   // decode kernel (steps: 64-wide K groups)
};

// Kernel and split choice.  The tile variant never changes an element's
// summation order; the split count (decode only) is a function of (N, K).
constexpr int SPLIT_MAX_M = DECODE_MAX_ROWS;

// Macro tile of the large-M kernel: 256 x 256 (16 waves), 192 x 256 (12
// waves) or 128 x 128 (8 waves of 64 x 32, two workgroups per CU; with four
// waves of 64 x 64 instead, one workgroup on a CU kept a single wave per
// SIMD and ran the flow expert's projections up to 13 % slower).  Each is priced as
// the number of rounds its tiles take over the stream's CUs times one round's
// work per CU, divided by the variant's throughput relative to 256 x 256
// (measured: 0.85 and 0.8); the cheapest wins, ties to the larger tile.  The
// smaller tiles pay off where 256 x 256 tiles leave most of a last round
// idle (e.g. 576 tiles = 2.25 rounds).  Every variant runs the same K loop,
// so an element's summation order does not depend on the choice.
static void big_tile(int M, int N, int cus, int& bm, int& bn) {
    const int CUS = cus;
    struct V { int bm, bn, per_cu; double rel; } vs[] = {{256, 256, 1, 1.0}, {192, 256, 1, 0.85}, {128, 128, 2, 0.8}};
    double best = 0;
    for (int i = 0; i < 3; ++i) {
        const V& v = vs[i];
        const long tiles = (long)((M + v.bm - 1) / v.bm) * ((N + v.bn - 1) / v.bn);
        const long rounds = (tiles + (long)CUS * v.per_cu - 1) / ((long)CUS * v.per_cu);
        const double cost = rounds * (double)v.bm * v.bn * v.per_cu / (65536.0 * v.rel);
        if (i == 0 || cost < best * 0.999) {
            best = cost;
            bm = v.bm;
            bn = v.bn;
        }
    }
}

static GemmPlan plan_gemm(bool bf16, int M, int N, int K, size_t ws_floats, bool split_ok, int cus = 256) {
    GemmPlan p;
    p.big = false;
    p.dec = false;
    p.bn = 0;
    p.splits = 1;
    p.k_per_split = K;
    if (bf16 && split_ok && K % 64 == 0) {
        // K splits: about 64 (column slice, split) pairs, each split at least
        // 16 K groups (1024 wide) -- the cross-workgroup hand-off costs about
        // as much as streaming that much more.  Narrow outputs with a long K
        // (at least 8192, e.g. a down projection of an 11008-wide MLP) aim for
        // about 256 pairs with splits of at least 512: measured 19-45 % more
        // bandwidth there at 1-64 rows, while shorter K lost by splitting
        // further.  A function of (N, K) only.  The partial tiles (up to four
        // row tiles, 32- or 64-column slices: at most 8 x tiles_n tiles) must
        // fit the workspace and counters.
        p.dec = true;
        const int tiles_n = (N + DEC_BN - 1) / DEC_BN;
        const int kgroups = K / 64;
        const int want = (tiles_n < 128 && kgroups >= 128)
                             ? std::min({(256 + tiles_n - 1) / tiles_n, kgroups / 8, DEC_MAX_SPLITS})
                             : std::max(1, std::min({(64 + tiles_n - 1) / tiles_n, kgroups / 16, DEC_MAX_SPLITS}));
        int gps = (kgroups + want - 1) / want;
        for (;;) {
            const int sp = (kgroups + gps - 1) / gps;
            if (sp == 1) break;
            if (sp <= DEC_MAX_SPLITS && (size_t)sp * 8 * tiles_n * DEC_TILE_FLOATS <= ws_floats &&
                8 * tiles_n <= DEC_MAX_COUNTERS)
                break;
            ++gps;
        }
        p.steps_per_split = gps;
        p.splits = (kgroups + gps - 1) / gps;
        // Row tiles of 16, 32 or 64 rows (any choice leaves every sum's
        // order unchanged): up to four row tiles when the column slices x
        // splits alone fill under half the chip -- each workgroup then
        // streams a quarter of the activations; otherwise the fewest tiles.
        if ((long)tiles_n * p.splits >= 128) p.tm = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
        else p.tm = M <= 64 ? 1 : (M <= 128 ? 2 : 4);
        p.m_tiles = (M + 16 * p.tm - 1) / (16 * p.tm);
        // 32-column slices when that still leaves under 3/4 of the CUs idle
        p.dbn = (long)tiles_n * p.splits * p.m_tiles < 3L * cus / 4 ? 32 : 64;
        // 96-column slices (fragment pairs stay whole; two LDS buffers) when
        // they take fewer rounds of one workgroup per CU: priced as rounds x
        // the bytes a workgroup streams per K element (weight plus
        // activation rows).  A CU's DMA stream runs at about the same rate
        // for either width, so the last, partly filled round is what the
        // wider slice saves: 7B-class gate/up (22016 outputs: 344 slices of
        // 64 = 1.34 rounds, 230 of 96 = one) measured 20-24 % faster at 1-32
        // rows; narrower outputs (one round either way) lose.  Row tiles of
        // 64 with 96 columns fill the LDS and leave no partial-tile stride
        // for K splits; smaller row tiles take 96 columns with one row tile
        // only.  The slice width never changes a sum's order.
        if (p.dbn == 64 && (p.tm == 4 ? p.splits == 1 : p.m_tiles == 1)) {
            auto cost = [&](int bn) {
                const long wgs = (long)((N + bn - 1) / bn) * p.splits * p.m_tiles;
                return ((wgs + cus - 1) / cus) * (bn + 16 * p.tm);
            };
            if (cost(96) < cost(64)) p.dbn = 96;
        }
        return p;
    }
    if (bf16 && !split_ok && M >= 256 && K % 64 == 0) {
        p.big = true;
        big_tile(M, N, cus, p.bm, p.bn);
        return p;
    }
    if (!bf16) p.bm = 64;
    else if (M <= 16) p.bm = 16;
    else if (M <= 32) p.bm = 32;
    else if (M <= 64) p.bm = 64;
    else p.bm = 128;
    if (!split_ok) return p;
    // one row of 128-wide column tiles -> enough K splits for ~512 workgroups
    const long tiles = (N + 127) / 128;
    int splits = 1;
    if (tiles < 256) {
        const int kblocks = (K + BK - 1) / BK;
        splits = (int)std::min<long>((512 + tiles - 1) / tiles, (long)std::max(1, kblocks / 2));
        splits = std::max(1, std::min(splits, 16));
    }
    while (splits > 1 && (size_t)splits * SPLIT_MAX_M * N > ws_floats) --splits;
    int kps = (K + splits - 1) / splits;
    kps = (kps + BK - 1) / BK * BK;
    p.splits = (K + kps - 1) / kps;
    p.k_per_split = kps;
    return p;
}

template <bool PAIRED, class Epi>
static void launch_bf16(const GemmArgs& a, const GemmPlan& p, Epi epi, hipStream_t s) {
    const bool split = p.splits > 1;
    if (p.big) {
        const long tiles = (long)((a.M + p.bm - 1) / p.bm) * ((a.N + p.bn - 1) / p.bn);
        dim3 grid((unsigned)tiles, 1);
        if (p.bm == 256)
            hipLaunchKernelGGL((gemm_bf16_big_kernel<256, 256, 4, 4, PAIRED, false, Epi>), grid, dim3(1024), 0, s,
                               (const bf16_t*)a.A, a.lda, (const bf16_t*)a.B, a.ldb, a.M, a.N, a.K, a.K, a.ws, epi);
        else if (p.bm == 192 && a.K >= 2048)
            hipLaunchKernelGGL((gemm_bf16_big_kernel<192, 256, 3, 4, PAIRED, true, Epi>), grid, dim3(768), 0, s,
                               (const bf16_t*)a.A, a.lda, (const bf16_t*)a.B, a.ldb, a.M, a.N, a.K, a.K, a.ws, epi);
        else if (p.bm == 192)
            hipLaunchKernelGGL((gemm_bf16_big_kernel<192, 256, 3, 4, PAIRED, false, Epi>), grid, dim3(768), 0, s,
                               (const bf16_t*)a.A, a.lda, (const bf16_t*)a.B, a.ldb, a.M, a.N, a.K, a.K, a.ws, epi);
        else
            hipLaunchKernelGGL((gemm_bf16_big_kernel<128, 128, 2, 4, PAIRED, true, Epi>), grid, dim3(512), 0, s,
                               (const bf16_t*)a.A, a.lda, (const bf16_t*)a.B, a.ldb, a.M, a.N, a.K, a.K, a.ws, epi);
        return;
    }
    if (p.dec) {
        auto godec = [&](auto kern, int bn) {
            dim3 grid(((a.N + bn - 1) / bn) * p.splits * p.m_tiles);
            hipLaunchKernelGGL(kern, grid, dim3(256), 0, s, (const bf16_t*)a.A, a.lda, (const bf16_t*)a.B,
                               a.ldb, a.M, a.N, a.K, p.steps_per_split, p.splits, p.m_tiles, a.ws,
                               a.counters, a.norm_eps, epi);
        };
        // Non-temporal weight loads where each weight slice is read by a
        // single workgroup (one row tile) of 64- or 96-column slices: measured 5-13 %
        // faster there, slower where row tiles or narrow slices re-read it.
        auto pick = [&](auto NORM) {
            constexpr bool NM = decltype(NORM)::value;
            if (p.dbn == 96) {   // row tiles of 16 or 32 rows: one tile (plan_gemm)
                if (p.tm == 1) godec(gemm_bf16_decode_kernel<1, 96, true, NM, PAIRED, Epi>, 96);
                else if (p.tm == 2) godec(gemm_bf16_decode_kernel<2, 96, true, NM, PAIRED, Epi>, 96);
                else if (p.m_tiles == 1) godec(gemm_bf16_decode_kernel<4, 96, true, NM, PAIRED, Epi>, 96);
                else godec(gemm_bf16_decode_kernel<4, 96, false, NM, PAIRED, Epi>, 96);
            } else if (p.dbn == 32) {
                if (p.tm == 1) godec(gemm_bf16_decode_kernel<1, 32, false, NM, PAIRED, Epi>, 32);
                else if (p.tm == 2) godec(gemm_bf16_decode_kernel<2, 32, false, NM, PAIRED, Epi>, 32);
                else godec(gemm_bf16_decode_kernel<4, 32, false, NM, PAIRED, Epi>, 32);
            } else if (p.m_tiles == 1) {
                if (p.tm == 1) godec(gemm_bf16_decode_kernel<1, 64, true, NM, PAIRED, Epi>, 64);
                else if (p.tm == 2) godec(gemm_bf16_decode_kernel<2, 64, true, NM, PAIRED, Epi>, 64);
                else godec(gemm_bf16_decode_kernel<4, 64, true, NM, PAIRED, Epi>, 64);
            } else {
                if (p.tm == 1) godec(gemm_bf16_decode_kernel<1, 64, false, NM, PAIRED, Epi>, 64);
                else if (p.tm == 2) godec(gemm_bf16_decode_kernel<2, 64, false, NM, PAIRED, Epi>, 64);
                else godec(gemm_bf16_decode_kernel<4, 64, false, NM, PAIRED, Epi>, 64);
            }
        };
        // the folded RMSNorm exists for the projections that follow a norm
        // (fused QKV, gate/up) and needs the whole K in one workgroup
        if constexpr (PAIRED) {
            if (a.row_norm && p.splits == 1) { pick(std::true_type{}); return; }
        }
        pick(std::false_type{});
        return;
    }
    auto go = [&](auto kern, int bm, int bn) {
        dim3 grid(((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn), p.splits);
        hipLaunchKernelGGL(kern, grid, dim3(256), 0, s, (const bf16_t*)a.A, a.lda,
                           (const bf16_t*)a.B, a.ldb, a.M, a.N, a.K, p.k_per_split, a.ws, epi);
    };
    switch (p.bm) {
    case 16:
        if (split) go(gemm_bf16_kernel<16, 256, 1, 4, PAIRED, true, Epi>, 16, 256);
        else go(gemm_bf16_kernel<16, 256, 1, 4, PAIRED, false, Epi>, 16, 256);
        break;
    case 32:
        if (split) go(gemm_bf16_kernel<32, 128, 1, 4, PAIRED, true, Epi>, 32, 128);
        else go(gemm_bf16_kernel<32, 128, 1, 4, PAIRED, false, Epi>, 32, 128);
        break;
    case 64:
        if (split) go(gemm_bf16_kernel<64, 128, 1, 4, PAIRED, true, Epi>, 64, 128);
        else go(gemm_bf16_kernel<64, 128, 1, 4, PAIRED, false, Epi>, 64, 128);
        break;
    default:
        if (split) go(gemm_bf16_kernel<128, 128, 2, 2, PAIRED, true, Epi>, 128, 128);
        else go(gemm_bf16_kernel<128, 128, 2, 2, PAIRED, false, Epi>, 128, 128);
        break;
    }
    if (split) {
        const int groups = PAIRED ? a.N / 8 : a.N / 4;
        long total = (long)a.M * groups;
        int blocks = (int)std::min<long>((total + 255) / 256, 4096);
        hipLaunchKernelGGL((splitk_reduce_kernel<PAIRED, Epi>), dim3(blocks), dim3(256), 0, s,
                           a.ws, p.splits, a.M, a.N, epi);
    }
}

template <bool PAIRED, class Epi>
static void launch_f32(const GemmArgs& a, const GemmPlan& p, Epi epi, hipStream_t s) {
    dim3 grid(((a.M + 63) / 64) * ((a.N + 63) / 64), p.splits);
    if (p.splits > 1) {
        hipLaunchKernelGGL((gemm_f32_kernel<PAIRED, true, Epi>), grid, dim3(256), 0, s,
                           (const float*)a.A, a.lda, (const float*)a.B, a.ldb, a.M, a.N, a.K,
                           p.k_per_split, a.ws, epi);
        const int groups = PAIRED ? a.N / 8 : a.N / 4;
        long total = (long)a.M * groups;
        int blocks = (int)std::min<long>((total + 255) / 256, 4096);
        hipLaunchKernelGGL((splitk_reduce_kernel<PAIRED, Epi>), dim3(blocks), dim3(256), 0, s,
                           a.ws, p.splits, a.M, a.N, epi);
    } else {
        hipLaunchKernelGGL((gemm_f32_kernel<PAIRED, false, Epi>), grid, dim3(256), 0, s,
                           (const float*)a.A, a.lda, (const float*)a.B, a.ldb, a.M, a.N, a.K,
                           p.k_per_split, a.ws, epi);
    }
}

template <bool PAIRED, class Epi>
static int dispatch(const GemmArgs& a, Epi epi, hipStream_t s) {
    const GemmPlan p = plan_gemm(a.bf16, a.M, a.N, a.K, a.ws_floats,
                                 a.split_ok && a.M <= SPLIT_MAX_M && (!a.bf16 || a.counters),
                                 std::max(1, std::min(a.cus, 256)));
    if (a.bf16) launch_bf16<PAIRED>(a, p, epi, s);
    else launch_f32<PAIRED>(a, p, epi, s);
    return p.splits;
}

int gemm(const GemmArgs& a, hipStream_t s) {
    if (a.M <= 0 || a.N <= 0) return 0;
    switch (a.epi) {
    case EPI_F32:
        return dispatch<false>(a, EpiF32{(float*)a.C, a.ldc}, s);
    case EPI_ACT:
        if (a.bf16) return dispatch<false>(a, EpiStore<bf16_t>{(bf16_t*)a.C, a.ldc}, s);
        return dispatch<false>(a, EpiStore<float>{(float*)a.C, a.ldc}, s);
    case EPI_RESID:
        return dispatch<false>(a, EpiResid{(float*)a.C, a.ldc, (bf16_t*)a.xb, a.ldxb}, s);
    case EPI_REMAP:
        if (a.bf16)
            return dispatch<false>(a, EpiRemap<bf16_t>{(float*)a.C, a.ldc, a.row_base, a.group,
                                                       (const bf16_t*)a.add, a.add_ld}, s);
        return dispatch<false>(a, EpiRemap<float>{(float*)a.C, a.ldc, a.row_base, a.group,
                                                  (const float*)a.add, a.add_ld}, s);
    case EPI_SWIGLU:
        if (a.bf16) return dispatch<true>(a, EpiSwiGLU<bf16_t>{(bf16_t*)a.C, a.ldc}, s);
        return dispatch<true>(a, EpiSwiGLU<float>{(float*)a.C, a.ldc}, s);
    case EPI_QKV:
        if (a.bf16) return dispatch<true>(a, make_epi_qkv<bf16_t>(*a.rope), s);
        return dispatch<true>(a, make_epi_qkv<float>(*a.rope), s);
    }
    return 0;
}

int gemm_splits(bool bf16, int M, int N, int K, size_t ws_floats, bool split_ok) {
    return plan_gemm(bf16, M, N, K, ws_floats, split_ok && M <= SPLIT_MAX_M).splits;
}

bool gemm_row_norm_ok(bool bf16, int M, int N, int K, size_t ws_floats) {
    if (!bf16 || M > SPLIT_MAX_M || K % 64) return false;
    const GemmPlan p = plan_gemm(true, M, N, K, ws_floats, true);
    return p.dec && p.splits == 1;
}

size_t gemm_counter_words() {
    return DEC_MAX_COUNTERS;
}

size_t gemm_ws_floats_used(bool bf16, int M, int N, int K, size_t ws_floats, bool split_ok) {
    const GemmPlan p = plan_gemm(bf16, M, N, K, ws_floats, split_ok && M <= SPLIT_MAX_M);
    if (p.splits <= 1) return 0;
    if (p.dec) return (size_t)((N + p.dbn - 1) / p.dbn) * p.m_tiles * p.splits * DEC_TILE_FLOATS;
    return (size_t)p.splits * M * N;
}

}  // namespace ebrl
