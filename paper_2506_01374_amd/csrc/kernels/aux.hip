// Auxiliary kernels of the contraction family: unfused epilogues, MoE
// routing preparation and the MoE weighted combine.
//
// Compile-time sizes (generated prologue):
//   EW_N          elements of an unfused elementwise epilogue
//   EW_COLS       columns of the bias + SiLU epilogue (bias length)
//   EW_SPLITS     K-split partial sums added by rc_splitk_sum_bf16 /
//                 rc_splitk_swiglu_bf16 (EW_N = rows x EW_COLS each, stored
//                 compact; the result goes to column EW_C0 + c of an output
//                 whose rows are EW_LD elements apart)
//   MOE_T MOE_TOPK MOE_E MOE_H   tokens, slots per token, experts, hidden
//   MOE_TM_UP MOE_TM_DOWN        M tiles of the two expert GEMMs

typedef unsigned short bf16_t;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16_t f2bf(float x) { return __builtin_bit_cast(bf16_t, (__bf16)x); }
__device__ __forceinline__ float bf2f(bf16_t b) {
    return __builtin_bit_cast(float, (unsigned)b << 16);
}
__device__ __forceinline__ float silu(float x) {
    return x / (1.0f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
}

struct EwArgs {
    const float *G;
    const float *U;
    const float *bias;
    bf16_t *out;
};

#ifdef EW_N
// out[i] = bf16(SiLU(G[i]) * U[i]), four elements per thread.
extern "C" __global__ __launch_bounds__(256) void rc_swiglu_f32(EwArgs a) {
    const long i = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= EW_N) return;
    f32x4 g = *(const f32x4 *)(a.G + i), u = *(const f32x4 *)(a.U + i);
    u32x2 p;
    p[0] = (unsigned)f2bf(silu(g[0]) * u[0]) | ((unsigned)f2bf(silu(g[1]) * u[1]) << 16);
    p[1] = (unsigned)f2bf(silu(g[2]) * u[2]) | ((unsigned)f2bf(silu(g[3]) * u[3]) << 16);
    *(u32x2 *)(a.out + i) = p;
}

// out[m][n] = bf16(SiLU(G[m][n] + bias[n])) (EW_ACT 1) or
// bf16(G[m][n] + bias[n]) (EW_ACT 0), four elements per thread.
#ifndef EW_ACT
#define EW_ACT 1
#endif
__device__ __forceinline__ float ew_act(float x) {
#if EW_ACT
    return silu(x);
#else
    return x;
#endif
}
extern "C" __global__ __launch_bounds__(256) void rc_bias_silu_f32(EwArgs a) {
    const long i = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= EW_N) return;
    const int n = (int)(i % EW_COLS);
    f32x4 g = *(const f32x4 *)(a.G + i);
    u32x2 p;
    p[0] = (unsigned)f2bf(ew_act(g[0] + a.bias[n])) | ((unsigned)f2bf(ew_act(g[1] + a.bias[n + 1])) << 16);
    p[1] = (unsigned)f2bf(ew_act(g[2] + a.bias[n + 2])) | ((unsigned)f2bf(ew_act(g[3] + a.bias[n + 3])) << 16);
    *(u32x2 *)(a.out + i) = p;
}

#ifdef EW_SPLITS
#ifndef EW_LD
#define EW_LD EW_COLS
#endif
#ifndef EW_C0
#define EW_C0 0
#endif
// Sums of the EW_SPLITS partial arrays at P[i] (8 consecutive elements of one
// row: EW_COLS is a multiple of 8), added in a fixed order.
__device__ __forceinline__ void splitk_sum8(const float *P, long i, f32x4 &s0, f32x4 &s1) {
    s0 = *(const f32x4 *)(P + i);
    s1 = *(const f32x4 *)(P + i + 4);
#pragma unroll
    for (int z = 1; z < EW_SPLITS; ++z) {
        s0 += *(const f32x4 *)(P + (long)z * EW_N + i);
        s1 += *(const f32x4 *)(P + (long)z * EW_N + i + 4);
    }
}
__device__ __forceinline__ long splitk_out(long i) {
    return (i / EW_COLS) * (long)EW_LD + EW_C0 + i % EW_COLS;
}

// out = bf16(G[0] + ... + G[EW_SPLITS - 1]): a GEMM whose K range was cut
// over EW_SPLITS workgroups; eight elements per thread.
extern "C" __global__ __launch_bounds__(256) void rc_splitk_sum_bf16(EwArgs a) {
    const long i = ((long)blockIdx.x * 256 + threadIdx.x) * 8;
    if (i >= EW_N) return;
    f32x4 s0, s1;
    splitk_sum8(a.G, i, s0, s1);
    u32x4 p;
    p[0] = (unsigned)f2bf(s0[0]) | ((unsigned)f2bf(s0[1]) << 16);
    p[1] = (unsigned)f2bf(s0[2]) | ((unsigned)f2bf(s0[3]) << 16);
    p[2] = (unsigned)f2bf(s1[0]) | ((unsigned)f2bf(s1[1]) << 16);
    p[3] = (unsigned)f2bf(s1[2]) | ((unsigned)f2bf(s1[3]) << 16);
    *(u32x4 *)(a.out + splitk_out(i)) = p;
}

// out = bf16(SiLU(sum of the G partials) * (sum of the U partials)): the
// gate and up products of a K-split gate/up GEMM; eight elements per thread.
extern "C" __global__ __launch_bounds__(256) void rc_splitk_swiglu_bf16(EwArgs a) {
    const long i = ((long)blockIdx.x * 256 + threadIdx.x) * 8;
    if (i >= EW_N) return;
    f32x4 g0, g1, u0, u1;
    splitk_sum8(a.G, i, g0, g1);
    splitk_sum8(a.U, i, u0, u1);
    u32x4 p;
    p[0] = (unsigned)f2bf(silu(g0[0]) * u0[0]) | ((unsigned)f2bf(silu(g0[1]) * u0[1]) << 16);
    p[1] = (unsigned)f2bf(silu(g0[2]) * u0[2]) | ((unsigned)f2bf(silu(g0[3]) * u0[3]) << 16);
    p[2] = (unsigned)f2bf(silu(g1[0]) * u1[0]) | ((unsigned)f2bf(silu(g1[1]) * u1[1]) << 16);
    p[3] = (unsigned)f2bf(silu(g1[2]) * u1[2]) | ((unsigned)f2bf(silu(g1[3]) * u1[3]) << 16);
    *(u32x4 *)(a.out + splitk_out(i)) = p;
}
#endif
#endif

#ifdef MOE_T
#define MOE_ROWS (MOE_T * MOE_TOPK)

// Routing preparation: a stable counting sort of the routed rows by expert
// in two kernels over blocks of PREP_T consecutive rows (one row per
// thread; expert ids out of range are clamped to expert 0 so that no write
// can leave its buffer).
//   rc_moe_hist: block b counts its rows per expert (LDS atomics) and
//     writes the counts to counts[b][*].
//   rc_moe_prep: block b reads the whole counts table; thread e sums
//     column e (all blocks: the expert's total; blocks before b: the rows
//     of expert e that precede this block).  A block-wide exclusive scan of
//     the totals gives offsets[] and, from ceil(count / tile), the tile
//     starts of both expert GEMMs (block 0 writes them).  Within the block,
//     the lanes of a wave holding the same expert are found with one
//     ballot per bit of the expert id, the lowest of them records the
//     group's size for its wave, and an exclusive prefix over the waves
//     gives each wave's first row per expert.  A row's permuted position is
//     offsets[e] + (rows of e in earlier blocks) + (rows of e in earlier
//     waves of the block) + (lanes of e below it in its wave): rows keep
//     their order within an expert, so the result is deterministic.
#define PREP_T 1024
#define PREP_W (PREP_T / 64)
#define PREP_NB ((MOE_ROWS + PREP_T - 1) / PREP_T)
#define PREP_BITS (MOE_E <= 1 ? 1 : 32 - __builtin_clz(MOE_E - 1))

struct MoeHistArgs {
    const int *ids;
    int *counts;           // [PREP_NB][E]
};

__device__ __forceinline__ int prep_id(const int *ids, int i) {
    if (i >= MOE_ROWS) return -1;
    const int x = ids[i];
    return (x < 0 || x >= MOE_E) ? 0 : x;
}

extern "C" __global__ __launch_bounds__(PREP_T) void rc_moe_hist(MoeHistArgs a) {
    __shared__ int hist[MOE_E];
    const int tid = threadIdx.x;
    const int x = prep_id(a.ids, blockIdx.x * PREP_T + tid);
    for (int e = tid; e < MOE_E; e += PREP_T) hist[e] = 0;
    __syncthreads();
    if (x >= 0) atomicAdd(&hist[x], 1);
    __syncthreads();
    for (int e = tid; e < MOE_E; e += PREP_T) a.counts[(size_t)blockIdx.x * MOE_E + e] = hist[e];
}

struct MoePrepArgs {
    const int *ids;        // [T][TOPK] expert of each (token, slot)
    const int *counts;     // [PREP_NB][E] rows per block and expert
    int *offsets;          // [E + 1] first permuted row of each expert
    int *perm;             // [T * TOPK] permuted row -> token * TOPK + slot
    int *pos;              // [T * TOPK] token * TOPK + slot -> permuted row
    int *tile_up;          // [E + 1] first M tile of each expert, up GEMM
    int *tile_down;        // [E + 1] first M tile of each expert, down GEMM
};

extern "C" __global__ __launch_bounds__(PREP_T) void rc_moe_prep(MoePrepArgs a) {
    __shared__ int wcnt[PREP_W][MOE_E];      // rows per (wave, expert), then first rows
    __shared__ int wsum[3][PREP_W];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, b = blockIdx.x;
    const int i = b * PREP_T + tid;
    const int x = prep_id(a.ids, i);
    for (int k = tid; k < PREP_W * MOE_E; k += PREP_T) (&wcnt[0][0])[k] = 0;

    // lanes of this wave holding the same expert
    const bool valid = x >= 0;
    unsigned long long m = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < PREP_BITS; ++bit) {
        const bool on = valid && ((x >> bit) & 1);
        const unsigned long long bb = __ballot(on);
        m &= on ? bb : ~bb;
    }
    const unsigned long long below = m & ((1ull << lane) - 1ull);
    __syncthreads();                          // wcnt cleared
    if (valid && below == 0ull) wcnt[wave][x] = __popcll(m);

    // expert totals and the rows of each expert in earlier blocks
    int h = 0, before = 0;
    if (tid < MOE_E) {
        int blk = 0;
        for (; blk + 8 <= PREP_NB; blk += 8) {
            int c[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) c[j] = a.counts[(size_t)(blk + j) * MOE_E + tid];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                h += c[j];
                before += (blk + j < b) ? c[j] : 0;
            }
        }
        for (; blk < PREP_NB; ++blk) {
            const int c = a.counts[(size_t)blk * MOE_E + tid];
            h += c;
            before += blk < b ? c : 0;
        }
    }
    const int hu = (h + MOE_TM_UP - 1) / MOE_TM_UP, hd = (h + MOE_TM_DOWN - 1) / MOE_TM_DOWN;
    int ih = h, iu = hu, id = hd;              // inclusive scans within the wave
    for (int d = 1; d < 64; d <<= 1) {
        const int th = __shfl_up(ih, d), tu = __shfl_up(iu, d), td = __shfl_up(id, d);
        if (lane >= d) { ih += th; iu += tu; id += td; }
    }
    if (lane == 63) { wsum[0][wave] = ih; wsum[1][wave] = iu; wsum[2][wave] = id; }
    __syncthreads();                          // wsum and the wave group sizes are in
    if (tid < MOE_E) {
        int bh = 0, bu = 0, bd = 0;
        for (int w = 0; w < wave; ++w) { bh += wsum[0][w]; bu += wsum[1][w]; bd += wsum[2][w]; }
        const int off = bh + ih - h;
        if (b == 0) {
            a.offsets[tid] = off;
            a.tile_up[tid] = bu + iu - hu;
            a.tile_down[tid] = bd + id - hd;
            if (tid == MOE_E - 1) {
                a.offsets[MOE_E] = bh + ih;
                a.tile_up[MOE_E] = bu + iu;
                a.tile_down[MOE_E] = bd + id;
            }
        }
        // first permuted row of each wave's rows of expert tid
        int run = off + before;
        for (int w = 0; w < PREP_W; ++w) {
            const int c = wcnt[w][tid];
            wcnt[w][tid] = run;
            run += c;
        }
    }
    __syncthreads();
    if (valid) {
        const int p = wcnt[wave][x] + __popcll(below);
        a.perm[p] = i;
        a.pos[i] = p;
    }
}

struct MoeCombineArgs {
    const bf16_t *Y;       // [T * TOPK][H] expert outputs in permuted order
    const int *pos;        // [T * TOPK]
    const float *w;        // [T][TOPK]
    bf16_t *out;           // [T][H]
};

// out[t][n] = bf16( sum_s w[t][s] * Y[pos[t * TOPK + s]][n] ), eight columns
// per thread, slots summed in order.
extern "C" __global__ __launch_bounds__(256) void rc_moe_combine(MoeCombineArgs a) {
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    const long cols = MOE_H / 8;
    if (idx >= (long)MOE_T * cols) return;
    const int t = (int)(idx / cols), n = (int)(idx % cols) * 8;
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
#pragma unroll
    for (int s = 0; s < MOE_TOPK; ++s) {
        const float ws = a.w[t * MOE_TOPK + s];
        const int p = a.pos[t * MOE_TOPK + s];
        u32x4 y = *(const u32x4 *)(a.Y + (size_t)p * MOE_H + n);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            acc[2 * j] += ws * bf2f((bf16_t)(y[j] & 0xFFFF));
            acc[2 * j + 1] += ws * bf2f((bf16_t)(y[j] >> 16));
        }
    }
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = (unsigned)f2bf(acc[2 * j]) | ((unsigned)f2bf(acc[2 * j + 1]) << 16);
    *(u32x4 *)(a.out + (size_t)t * MOE_H + n) = o;
}
#endif
