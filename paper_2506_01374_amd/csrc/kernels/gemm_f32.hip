// fp32 GEMM C[M][N] = A[M][K] B[K][N] on gfx950 with v_mfma_f32_16x16x4_f32
// (the fp32 contraction of the paper's App. A example module).
//
// Compile-time schedule (defined by the generated prologue):
//   TM TN TK     workgroup tile (TileSize)
//   WM WN        waves per workgroup along M and N (Parallel)
//   VEC          fp32 elements per global load (Vectorize)
//   STAGES       1: load-store-compute; 2: LDS double buffer with register
//                prefetch of the next K tile (ComputeLocation); 3: streaming
//                for decode-shaped operators (M <= 16 rows, one MFMA row
//                block): no LDS staging, each wave streams its own slice of
//                the K range straight from memory into MFMA operands with
//                the loads of the next 2 x UNROLL - 1 batches of TK rows in
//                flight (Unroll sets the prefetch depth), the waves' partial sums
//                are added in LDS, and with SPLITS > 1 the workgroups of one
//                column tile split K further and rc_gemm_f32_splitk_reduce
//                adds their partials (in a fixed order)
//   SPLITS       K splits across workgroups (Parallel; STAGES 3 only)
//   UNROLL       unroll factor of the K-tile loop (Unroll)
//   LAYOUT       0: B stored [K][N]; 1: B stored [N][K] (Layout)
//   GM GN GK     problem size.  Stages 1 and 2 take any size: tiles that
//                cross the edge of M, N or K load zeros there and store only
//                inside C (VEC divides the row lengths, so a vector is wholly
//                inside or outside); a problem that every tile divides
//                compiles without the guards.  Stage 3 needs whole tiles.
//
// MFMA lane layout (16x16x4, one block): lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; accumulator element r of lane l is
// C[4 * (l / 16) + r][l % 16].

#define NT (64 * WM * WN)
#define WTM (TM / WM)
#define WTN (TN / WN)
#define FM (WTM / 16)
#define FN (WTN / 16)
#define KTILES ((GK + TK - 1) / TK)
#define RAGGED ((GM % TM) != 0 || (GN % TN) != 0 || (GK % TK) != 0)
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
    float *P;          // per-split partial sums [SPLITS][GM][GN] (STAGES 3, SPLITS > 1)
};

__device__ __forceinline__ float vget(const vecT &v, int j) {
#if VEC == 1
    (void)j;
    return v;
#else
    return v[j];
#endif
}

#if STAGES == 3
// Streaming variant.  Workgroup (nt, s) owns columns nt * 64 .. + 63 and the
// s-th of SPLITS equal K ranges; wave w of its NT / 64 waves takes the w-th
// slice of that range, KW rows, in batches of TK rows.
//
// Lane layout of one 16-row block kb .. kb + 15 (k-step e = 0..3 contracts
// the rows kb + 4 q + e, q = lane / 16 being the MFMA's k slot, so that A
// and B agree on which row each slot holds):
//   A: one 16-byte load per lane, A[lane % 16][kb + 4 q .. + 3]; element e
//      is the lane's A operand of k-step e (rows >= GM read as zero)
//   B: for each e one 16-byte load per lane, B[kb + 4 q + e][n0 + 4 c .. + 3]
//      with c = lane % 16; element j is the lane's B operand of the MFMA for
//      column group j (output columns n0 + 4 c + j)
// Accumulator j, element r of lane l is C[4 (l / 16) + r][n0 + 4 (l % 16) + j]:
// for each r a lane owns four consecutive columns.
#define SWAVES (WM * WN)
#define KSPLIT (GK / SPLITS)
#define KW (KSPLIT / SWAVES)
#define NBATCH (KW / TK)
#define BLK (TK / 16)

extern "C" __global__ __launch_bounds__(NT) void rc_gemm_f32(GemmF32Args args) {
    __shared__ f32x4 red[SWAVES][4][64];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ntn = GN / 64;
    const int nt = blockIdx.x % ntn, sp = blockIdx.x / ntn;
    const int n0 = nt * 64;
    const int k_first = sp * KSPLIT + wave * KW;
    const int q = lane >> 4, c = lane & 15;
    const bool arow = c < GM;
    const float *Arow = args.A + (size_t)(arow ? c : 0) * GK + 4 * q;
    const float *Bcol = args.B + (size_t)(4 * q) * GN + n0 + 4 * c;

    f32x4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Ring of PF register sets: the loads of the next PF - 1 batches are in
    // flight while a batch is multiplied (PF = 2 x UNROLL, at most NBATCH).
    constexpr int PF = (2 * UNROLL < NBATCH) ? 2 * UNROLL : NBATCH;
    f32x4 ra[PF][BLK], rb[PF][BLK][4];
    auto load = [&](int k0, int set) {
#pragma unroll
        for (int b = 0; b < BLK; ++b) {
            const int kb = k0 + 16 * b;
            ra[set][b] = arow ? *(const f32x4 *)(Arow + kb) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int e = 0; e < 4; ++e) rb[set][b][e] = *(const f32x4 *)(Bcol + (size_t)(kb + e) * GN);
        }
    };
    auto compute = [&](int set) {
#pragma unroll
        for (int b = 0; b < BLK; ++b)
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ra[set][b][e], rb[set][b][e][j], acc[j], 0, 0, 0);
    };
#pragma unroll
    for (int p = 0; p < PF; ++p) load(k_first + p * TK, p);
    for (int i = 0; i < NBATCH; i += PF) {
#pragma unroll
        for (int p = 0; p < PF; ++p) {
            if (i + p < NBATCH) {
                compute(p);
                if (i + p + PF < NBATCH) load(k_first + (i + p + PF) * TK, p);
            }
        }
    }

    // add the waves' partial sums in wave order
    if (SWAVES > 1) {
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][r][lane] = f32x4{acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            f32x4 v = red[0][r][lane];
#pragma unroll
            for (int w = 1; w < SWAVES; ++w) v += red[w][r][lane];
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[j][r] = v[j];
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int m = 4 * q + r;
        if (m >= GM) continue;
        const f32x4 v = f32x4{acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
#if SPLITS == 1
        *(f32x4 *)(args.C + (size_t)m * GN + n0 + 4 * c) = v;
#else
        *(f32x4 *)(args.P + ((size_t)sp * GM + m) * GN + n0 + 4 * c) = v;
#endif
    }
}

#if SPLITS > 1
// C = sum over splits of the partials in a fixed association: each of four
// threads per 4-column group sums the splits g, g + 4, g + 8, ... in order
// and the four group sums are added in group order through LDS.  A
// workgroup covers 64 four-column groups.
extern "C" __global__ __launch_bounds__(256) void rc_gemm_f32_splitk_reduce(GemmF32Args args) {
    __shared__ f32x4 part[4][64];
    const int t = threadIdx.x, g = t >> 6;
    const size_t i = (size_t)blockIdx.x * 64 + (t & 63);
    const bool ok = i < (size_t)GM * GN / 4;
    f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
    if (ok) {
#pragma unroll
        for (int s = g; s < SPLITS; s += 4) v += *(const f32x4 *)(args.P + (size_t)s * GM * GN + 4 * i);
    }
    part[g][t & 63] = v;
    __syncthreads();
    if (g == 0 && ok) *(f32x4 *)(args.C + 4 * i) = ((part[0][t] + part[1][t]) + part[2][t]) + part[3][t];
}
#endif

#else
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

    // a vector load of row `row`, columns col .. col + VEC - 1 of a
    // rows x cols matrix; zeros outside it (tiles crossing an edge)
    auto ld = [&](const float *base, int row, int col, int rows, int cols) -> vecT {
        if (RAGGED && (row >= rows || col >= cols)) return vecT{};
        return *(const vecT *)(base + (size_t)row * cols + col);
    };
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            int v = tid + i * NT;
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
            ra[i] = ld(args.A, m0 + r, k0 + c, GM, GK);
        }
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            int v = tid + i * NT;
#if LAYOUT == 0
            int r = v / (TN / VEC), c = (v % (TN / VEC)) * VEC;
            rb[i] = ld(args.B, k0 + r, n0 + c, GK, GN);
#else
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
            rb[i] = ld(args.B, n0 + r, k0 + c, GN, GK);
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
                if (!RAGGED || (m < GM && n < GN)) args.C[(size_t)m * GN + n] = acc[i][j][r];
            }
}
#endif
