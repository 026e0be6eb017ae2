// fp32 GEMM C[M][N] = A[M][K] B[K][N] on gfx950 with v_mfma_f32_16x16x4_f32
// (the fp32 contraction of the paper's App. A example module).
//
// Compile-time schedule (defined by the generated prologue):
//   TM TN TK     workgroup tile (TileSize)
//   WM WN        waves per workgroup along M and N (Parallel)
//   VEC          fp32 elements per global load (Vectorize)
//   STAGES       1: load-store-compute; 2: LDS double buffer with register
//                prefetch of the next K tile (ComputeLocation)
//   UNROLL       unroll factor of the K-tile loop (Unroll)
//   LAYOUT       0: B stored [K][N]; 1: B stored [N][K] (Layout)
//   GM GN GK     problem size; every tile is perfect (checked on the host).
//
// MFMA lane layout (16x16x4, one block): lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; accumulator element r of lane l is
// C[4 * (l / 16) + r][l % 16].

#define NT (64 * WM * WN)
#define WTM (TM / WM)
#define WTN (TN / WN)
#define FM (WTM / 16)
#define FN (WTN / 16)
#define KTILES (GK / TK)
#define A_LOADS ((TM * TK) / (VEC * NT))
#define B_LOADS ((TK * TN) / (VEC * NT))

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int V> struct FVec;
template <> struct FVec<1> { typedef float T; };
template <> struct FVec<2> { typedef float __attribute__((ext_vector_type(2))) T; };
template <> struct FVec<4> { typedef float __attribute__((ext_vector_type(4))) T; };
typedef typename FVec<VEC>::T vecT;

struct GemmF32Args {
    const float *A;
    const float *B;
    float *C;
};

__device__ __forceinline__ float vget(const vecT &v, int j) {
#if VEC == 1
    (void)j;
    return v;
#else
    return v[j];
#endif
}

extern "C" __global__ __launch_bounds__(NT) void rc_gemm_f32(GemmF32Args args) {
    __shared__ float As[STAGES][TM][TK + 1];
    __shared__ float Bs[STAGES][TK][TN + 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    vecT ra[A_LOADS], rb[B_LOADS];

    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            int v = tid + i * NT;
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
            ra[i] = *(const vecT *)(args.A + (size_t)(m0 + r) * GK + k0 + c);
        }
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            int v = tid + i * NT;
#if LAYOUT == 0
            int r = v / (TN / VEC), c = (v % (TN / VEC)) * VEC;
            rb[i] = *(const vecT *)(args.B + (size_t)(k0 + r) * GN + n0 + c);
#else
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
            rb[i] = *(const vecT *)(args.B + (size_t)(n0 + r) * GK + k0 + c);
#endif
        }
    };

    auto swrite = [&](int s) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            int v = tid + i * NT;
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
#pragma unroll
            for (int j = 0; j < VEC; ++j) As[s][r][c + j] = vget(ra[i], j);
        }
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            int v = tid + i * NT;
#if LAYOUT == 0
            int r = v / (TN / VEC), c = (v % (TN / VEC)) * VEC;
#pragma unroll
            for (int j = 0; j < VEC; ++j) Bs[s][r][c + j] = vget(rb[i], j);
#else
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
#pragma unroll
            for (int j = 0; j < VEC; ++j) Bs[s][c + j][r] = vget(rb[i], j);
#endif
        }
    };

    auto compute = [&](int s) {
#pragma unroll
        for (int kk = 0; kk < TK; kk += 4) {
            float a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) a[i] = As[s][wm * WTM + i * 16 + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
            for (int j = 0; j < FN; ++j) b[j] = Bs[s][kk + (lane >> 4)][wn * WTN + j * 16 + (lane & 15)];
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    };

#if STAGES == 1
#pragma unroll UNROLL
    for (int kt = 0; kt < KTILES; ++kt) {
        gload(kt * TK);
        swrite(0);
        __syncthreads();
        compute(0);
        __syncthreads();
    }
#else
    gload(0);
    swrite(0);
    __syncthreads();
#pragma unroll UNROLL
    for (int kt = 0; kt < KTILES; ++kt) {
        if (kt + 1 < KTILES) gload((kt + 1) * TK);
        compute(kt & 1);
        if (kt + 1 < KTILES) swrite((kt + 1) & 1);
        __syncthreads();
    }
#endif

#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int m = m0 + wm * WTM + i * 16 + 4 * (lane >> 4) + r;
                int n = n0 + wn * WTN + j * 16 + (lane & 15);
                args.C[(size_t)m * GN + n] = acc[i][j][r];
            }
}
