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

// Grid: MOE_E workgroups of 256 threads.  Every workgroup builds the full
// expert histogram in LDS (ids out of range are clamped to expert 0 so that
// no write can leave its buffer), derives the exclusive prefix offsets and
// the per-expert tile starts, and then workgroup e writes the rows routed to
// expert e in token order (a stable counting sort).  Workgroup 0 also
// publishes offsets and tile starts.
extern "C" __global__ __launch_bounds__(256) void rc_moe_prep(MoePrepArgs a) {
    __shared__ int hist[MOE_E];
    __shared__ int offs[MOE_E + 1];
    __shared__ int wave_cnt[4];
    const int tid = threadIdx.x, e = blockIdx.x;
    for (int i = tid; i < MOE_E; i += 256) hist[i] = 0;
    __syncthreads();
    for (int i = tid; i < MOE_ROWS; i += 256) {
        int x = a.ids[i];
        x = (x < 0 || x >= MOE_E) ? 0 : x;
        atomicAdd(&hist[x], 1);
    }
    __syncthreads();
    if (tid == 0) {
        int s = 0, tu = 0, td = 0;
        for (int x = 0; x < MOE_E; ++x) {
            offs[x] = s;
            if (e == 0) {
                a.offsets[x] = s;
                a.tile_up[x] = tu;
                a.tile_down[x] = td;
            }
            s += hist[x];
            tu += (hist[x] + MOE_TM_UP - 1) / MOE_TM_UP;
            td += (hist[x] + MOE_TM_DOWN - 1) / MOE_TM_DOWN;
        }
        offs[MOE_E] = s;
        if (e == 0) {
            a.offsets[MOE_E] = s;
            a.tile_up[MOE_E] = tu;
            a.tile_down[MOE_E] = td;
        }
    }
    __syncthreads();
    int base = offs[e];
    const int lane = tid & 63, wave = tid >> 6;
    for (int c0 = 0; c0 < MOE_ROWS; c0 += 256) {
        int i = c0 + tid;
        int x = i < MOE_ROWS ? a.ids[i] : -1;
        if (i < MOE_ROWS && (x < 0 || x >= MOE_E)) x = 0;
        bool hit = (x == e);
        unsigned long long ballot = __ballot(hit);
        int before = __popcll(ballot & ((1ull << lane) - 1ull));
        if (lane == 0) wave_cnt[wave] = __popcll(ballot);
        __syncthreads();
        int wbase = 0;
        for (int w = 0; w < wave; ++w) wbase += wave_cnt[w];
        int total = wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3];
        if (hit) {
            int p = base + wbase + before;
            a.perm[p] = i;
            a.pos[i] = p;
        }
        base += total;
        __syncthreads();
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
