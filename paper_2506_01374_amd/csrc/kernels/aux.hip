// Auxiliary kernels of the contraction family: unfused epilogues, MoE
// routing preparation and the MoE weighted combine.
//
// Compile-time sizes (generated prologue):
//   EW_N          elements of an unfused elementwise epilogue
//   EW_COLS       columns of the bias + SiLU epilogue (bias length)
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

// out[m][n] = bf16(SiLU(G[m][n] + bias[n])), four elements per thread.
extern "C" __global__ __launch_bounds__(256) void rc_bias_silu_f32(EwArgs a) {
    const long i = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= EW_N) return;
    const int n = (int)(i % EW_COLS);
    f32x4 g = *(const f32x4 *)(a.G + i);
    u32x2 p;
    p[0] = (unsigned)f2bf(silu(g[0] + a.bias[n])) | ((unsigned)f2bf(silu(g[1] + a.bias[n + 1])) << 16);
    p[1] = (unsigned)f2bf(silu(g[2] + a.bias[n + 2])) | ((unsigned)f2bf(silu(g[3] + a.bias[n + 3])) << 16);
    *(u32x2 *)(a.out + i) = p;
}
#endif

#ifdef MOE_T
#define MOE_ROWS (MOE_T * MOE_TOPK)

struct MoePrepArgs {
    const int *ids;        // [T][TOPK] expert of each (token, slot)
    int *offsets;          // [E + 1] first permuted row of each expert
    int *perm;             // [T * TOPK] permuted row -> token * TOPK + slot
    int *pos;              // [T * TOPK] token * TOPK + slot -> permuted row
    int *tile_up;          // [E + 1] first M tile of each expert, up GEMM
    int *tile_down;        // [E + 1] first M tile of each expert, down GEMM
};

// Grid: MOE_E workgroups of PREP_T threads.  Every workgroup copies all
// expert ids into LDS (ids out of range are clamped to expert 0 so that no
// write can leave its buffer), builds the expert histogram from per-wave
// sub-histograms, derives the exclusive prefix offsets and the per-expert
// tile starts, and then workgroup e writes the rows routed to expert e in
// token order (a stable counting sort): each thread owns a contiguous chunk
// of entries, counts its hits, and one block-wide exclusive scan of those
// counts gives every thread its first output row.  Workgroup 0 also
// publishes offsets and tile starts.
#define PREP_T 1024
#define PREP_W (PREP_T / 64)
#define PREP_CHUNK ((MOE_ROWS + PREP_T - 1) / PREP_T)

extern "C" __global__ __launch_bounds__(PREP_T) void rc_moe_prep(MoePrepArgs a) {
    __shared__ int ids[PREP_CHUNK * PREP_T];
    __shared__ int sub[PREP_W][MOE_E];
    __shared__ int offs[MOE_E + 1];
    __shared__ int wsum[PREP_W];
    const int tid = threadIdx.x, e = blockIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < PREP_W * MOE_E; i += PREP_T) (&sub[0][0])[i] = 0;
    for (int i = tid; i < PREP_CHUNK * PREP_T; i += PREP_T) {
        int x = i < MOE_ROWS ? a.ids[i] : -1;
        if (i < MOE_ROWS && (x < 0 || x >= MOE_E)) x = 0;
        ids[i] = x;
    }
    __syncthreads();
    for (int i = tid; i < MOE_ROWS; i += PREP_T) atomicAdd(&sub[wave][ids[i]], 1);
    __syncthreads();
    if (wave == 0) {
        // lane x sums expert x over the sub-histograms; one wave scans 64 bins
        int run = 0, tu = 0, td = 0;
        for (int base = 0; base < MOE_E; base += 64) {
            int x = base + lane;
            int h = 0;
            if (x < MOE_E)
                for (int w = 0; w < PREP_W; ++w) h += sub[w][x];
            int hu = (h + MOE_TM_UP - 1) / MOE_TM_UP, hd = (h + MOE_TM_DOWN - 1) / MOE_TM_DOWN;
            int ih = h, iu = hu, id = hd;          // inclusive scans across the wave
            for (int d = 1; d < 64; d <<= 1) {
                int th = __shfl_up(ih, d), tu2 = __shfl_up(iu, d), td2 = __shfl_up(id, d);
                if (lane >= d) { ih += th; iu += tu2; id += td2; }
            }
            if (x < MOE_E) {
                offs[x] = run + ih - h;
                if (e == 0) {
                    a.offsets[x] = run + ih - h;
                    a.tile_up[x] = tu + iu - hu;
                    a.tile_down[x] = td + id - hd;
                }
            }
            run += __shfl(ih, 63);
            tu += __shfl(iu, 63);
            td += __shfl(id, 63);
        }
        if (lane == 0) {
            offs[MOE_E] = run;
            if (e == 0) {
                a.offsets[MOE_E] = run;
                a.tile_up[MOE_E] = tu;
                a.tile_down[MOE_E] = td;
            }
        }
    }
    __syncthreads();
    // stable compaction of the entries routed to expert e
    const int c0 = tid * PREP_CHUNK;
    int cnt = 0;
    for (int j = 0; j < PREP_CHUNK; ++j) cnt += (c0 + j < MOE_ROWS && ids[c0 + j] == e);
    int inc = cnt;
    for (int d = 1; d < 64; d <<= 1) {
        int t = __shfl_up(inc, d);
        if (lane >= d) inc += t;
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    int p = offs[e] + before + inc - cnt;
    for (int j = 0; j < PREP_CHUNK; ++j) {
        int i = c0 + j;
        if (i < MOE_ROWS && ids[i] == e) {
            a.perm[p] = i;
            a.pos[i] = p;
            ++p;
        }
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
