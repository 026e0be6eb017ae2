// Softmax attention forward for gfx950, bf16 Q/K/V/O [B][H][S][D], fp32
// scores, online (blockwise) softmax, bf16 MFMA for both products.
//
// Compile-time schedule (generated prologue):
//   BM           query rows per workgroup (TileSize)
//   BN           keys per tile (TileSize)
//   NW           waves per workgroup; each owns BM / NW query rows (Parallel)
//   MF           MFMA shape 16 (16x16x32) or 32 (32x32x16)
//   STAGES       1: load tile, compute; 2: double-buffered K/V tiles with
//                register prefetch of the next tile (ComputeLocation)
//   VEC          bf16 per global load of K (Vectorize)
//   UNROLL       unroll factor of the key-tile loop (Unroll)
//   ORDER        0: query tiles in order; 1: longest (last) query tiles
//                first; 2: paired - workgroup b and b + half take query
//                tiles t and NQT-1-t, so that co-resident pairs carry equal
//                causal work
//   OCC          waves per SIMD the register allocation must leave room for
//   AB AH AS AD  batch, heads, sequence length, head dim
//   CAUSAL       top-left aligned causal mask (key j visible iff j <= i)
//   SCALE_LOG2   log2(e) / sqrt(AD): scores are kept in log2 units
//
// Layout of the products.  Scores are computed transposed, S^T = K Q^T,
// with K as the first MFMA operand: each lane then holds the scores of ONE
// query (column lane % MF) for several keys, so the softmax statistics
// (running max m and sum l) are per-lane scalars and the rescale of the
// output accumulator is a scalar multiply.  The output is accumulated
// transposed too, O^T = V^T P^T, with V^T fragments from an LDS copy of
// the V tile stored d-major; the probabilities never leave registers: the
// MFMA's k index (the key) follows the accumulator layout of S^T, and the
// V^T fragment is read in that same key order.

#define RPW (BM / NW)
#define QB (RPW / MF)
#define NT (64 * NW)
#define KB (BN / MF)
#define DB (AD / MF)
#define NQT (AS / BM)
#define CPR (AD / 8)
#define RPL ((16 / CPR) > 0 ? (16 / CPR) : 1)
#define VTS (BN + 4)
#define K_LOADS ((BN * AD / VEC + NT - 1) / NT)
#define V_BLKS ((BN * AD / 32 + NT - 1) / NT)

typedef unsigned short bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#if MF == 16
typedef f32x4 accT;
#define ACCN 4
#define KSTEP 32
#else
typedef f32x16 accT;
#define ACCN 16
#define KSTEP 16
#endif

template <int V> struct BVec;
template <> struct BVec<2> { typedef unsigned int T; };
template <> struct BVec<4> { typedef u32x2 T; };
template <> struct BVec<8> { typedef u32x4 T; };
typedef typename BVec<VEC>::T vecT;

struct AttnArgs {
    const bf16_t *Q;
    const bf16_t *K;
    const bf16_t *V;
    bf16_t *O;
};

__device__ __forceinline__ int kswz(int row, int chunk) {
    return row * AD + ((chunk ^ ((row / RPL) % CPR)) << 3);
}

__device__ __forceinline__ accT mfma(const bf16x8 &a, const bf16x8 &b, const accT &c) {
#if MF == 16
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
#else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
#endif
}

__device__ __forceinline__ unsigned pack2(float a, float b) {
    return (unsigned)__builtin_bit_cast(bf16_t, (__bf16)a) |
           ((unsigned)__builtin_bit_cast(bf16_t, (__bf16)b) << 16);
}

// Key offset (within an MF-key block) of accumulator element r of `lane`.
__device__ __forceinline__ int key_of(int r, int lane) {
#if MF == 16
    return 4 * (lane >> 4) + r;
#else
    return (r >> 2) * 8 + 4 * (lane >> 5) + (r & 3);
#endif
}

__device__ __forceinline__ float group_max(float v) {
#if MF == 16
    v = fmaxf(v, __shfl_xor(v, 16));
#endif
    return fmaxf(v, __shfl_xor(v, 32));
}

__device__ __forceinline__ float group_sum(float v) {
#if MF == 16
    v += __shfl_xor(v, 16);
#endif
    return v + __shfl_xor(v, 32);
}

extern "C" __global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
void rc_attention(AttnArgs args) {
    __shared__ __attribute__((aligned(16))) bf16_t Ks[STAGES][BN * AD];
    __shared__ __attribute__((aligned(16))) bf16_t Vt[STAGES][AD * VTS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bid = blockIdx.x;
#if ORDER == 1
    const int qt = NQT - 1 - bid / (AB * AH);
    const int bh = bid % (AB * AH);
#elif ORDER == 2
    const int half = (NQT / 2) * AB * AH;
    const int qt = bid < half ? NQT - 1 - bid / (AB * AH) : (bid - half) / (AB * AH);
    const int bh = bid % (AB * AH);
#else
    const int qt = bid % NQT;
    const int bh = bid / NQT;
#endif
    const int q0 = qt * BM;
    const int q0w = q0 + wave * RPW;
    const size_t base = (size_t)bh * AS * AD;

    bf16x8 qf[QB][AD / KSTEP];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int ks = 0; ks < AD / KSTEP; ++ks)
            qf[qb][ks] = *(const bf16x8 *)(args.Q + base + (size_t)(q0w + qb * MF + lane % MF) * AD +
                                           ks * KSTEP + 8 * (lane / MF));

    accT o[QB][DB];
    float m[QB], l[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m[qb] = -__builtin_inff();
        l[qb] = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < ACCN; ++r) o[qb][db][r] = 0.f;
    }

#if CAUSAL
    const int n_kt = (q0 + BM - 1) / BN + 1;
#else
    const int n_kt = AS / BN;
#endif

    vecT rk[K_LOADS];
    u32x4 rv[V_BLKS][4];

    auto gload = [&](int kt) {
        const bf16_t *Kg = args.K + base + (size_t)kt * BN * AD;
        const bf16_t *Vg = args.V + base + (size_t)kt * BN * AD;
#pragma unroll
        for (int i = 0; i < K_LOADS; ++i) {
            int idx = tid + i * NT;
            if (idx < BN * AD / VEC) rk[i] = *(const vecT *)(Kg + (size_t)idx * VEC);
        }
#pragma unroll
        for (int i = 0; i < V_BLKS; ++i) {
            int blk = tid + i * NT;
            if (blk < BN * AD / 32) {
                int kr = (blk / (AD / 8)) * 4, dc = (blk % (AD / 8)) * 8;
#pragma unroll
                for (int j = 0; j < 4; ++j) rv[i][j] = *(const u32x4 *)(Vg + (size_t)(kr + j) * AD + dc);
            }
        }
    };

    auto swrite = [&](int s) {
#pragma unroll
        for (int i = 0; i < K_LOADS; ++i) {
            int idx = tid + i * NT;
            if (idx < BN * AD / VEC) {
                int row = idx / (AD / VEC), c = (idx % (AD / VEC)) * VEC;
                *(vecT *)(Ks[s] + kswz(row, c >> 3) + (c & 7)) = rk[i];
            }
        }
#pragma unroll
        for (int i = 0; i < V_BLKS; ++i) {
            int blk = tid + i * NT;
            if (blk < BN * AD / 32) {
                int kr = (blk / (AD / 8)) * 4, dc = (blk % (AD / 8)) * 8;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    // column d = dc + j of keys kr .. kr+3
                    unsigned h[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) h[t] = (rv[i][t][j >> 1] >> (16 * (j & 1))) & 0xFFFF;
                    u32x2 w;
                    w[0] = h[0] | (h[1] << 16);
                    w[1] = h[2] | (h[3] << 16);
                    *(u32x2 *)(Vt[s] + (dc + j) * VTS + kr) = w;
                }
            }
        }
    };

    auto compute = [&](int kt, int s) {
#if CAUSAL
        if (kt * BN > q0w + RPW - 1) return;     // every key of the tile is masked for this wave
#endif
        // S^T = K Q^T for every query block; each K fragment is read once
        accT sc[QB][KB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) sc[qb][kb][r] = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int ks = 0; ks < AD / KSTEP; ++ks) {
                bf16x8 kf = *(const bf16x8 *)(Ks[s] + kswz(kb * MF + lane % MF, ks * (KSTEP / 8) + lane / MF));
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) sc[qb][kb] = mfma(kf, qf[qb][ks], sc[qb][kb]);
            }
        // online softmax, one query per lane; m is kept in log2 units and the
        // scale is folded into the exponent's fused multiply-add
#if CAUSAL
        // only a tile that crosses this wave's diagonal needs the mask
        const bool diag = kt * BN + BN - 1 > q0w;
#endif
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float mx = -__builtin_inff();
#if CAUSAL
            if (diag) {
                const int q = q0w + qb * MF + lane % MF;
#pragma unroll
                for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                    for (int r = 0; r < ACCN; ++r)
                        if (kt * BN + kb * MF + key_of(r, lane) > q) sc[qb][kb][r] = -__builtin_inff();
            }
#endif
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) mx = fmaxf(mx, sc[qb][kb][r]);
            mx = group_max(mx);
            const float mnew = fmaxf(m[qb], mx * SCALE_LOG2);
            const float alpha = __builtin_amdgcn_exp2f(m[qb] - mnew);
            float ps = 0.f;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) {
                    float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][kb][r], SCALE_LOG2, -mnew));
                    sc[qb][kb][r] = p;
                    ps += p;
                }
            ps = group_sum(ps);
            l[qb] = l[qb] * alpha + ps;
            m[qb] = mnew;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) o[qb][db][r] *= alpha;
        }
        // O^T += V^T P^T, KSTEP keys per MFMA; each V^T fragment is read once
#pragma unroll
        for (int j = 0; j < BN / KSTEP; ++j) {
            bf16x8 pf[QB];
#if MF == 16
            const int c0 = 32 * j + 4 * (lane >> 4), c1 = c0 + 16;
#else
            const int kb = j >> 1, hf = (j & 1) * 8;
            const int c0 = kb * 32 + (j & 1) * 16 + 4 * (lane >> 5), c1 = c0 + 8;
#endif
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                u32x4 pw;
#if MF == 16
                pw[0] = pack2(sc[qb][2 * j][0], sc[qb][2 * j][1]);
                pw[1] = pack2(sc[qb][2 * j][2], sc[qb][2 * j][3]);
                pw[2] = pack2(sc[qb][2 * j + 1][0], sc[qb][2 * j + 1][1]);
                pw[3] = pack2(sc[qb][2 * j + 1][2], sc[qb][2 * j + 1][3]);
#else
                pw[0] = pack2(sc[qb][kb][hf + 0], sc[qb][kb][hf + 1]);
                pw[1] = pack2(sc[qb][kb][hf + 2], sc[qb][kb][hf + 3]);
                pw[2] = pack2(sc[qb][kb][hf + 4], sc[qb][kb][hf + 5]);
                pw[3] = pack2(sc[qb][kb][hf + 6], sc[qb][kb][hf + 7]);
#endif
                pf[qb] = __builtin_bit_cast(bf16x8, pw);
            }
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int drow = db * MF + lane % MF;
                u32x4 vw;
                u32x2 a = *(const u32x2 *)(Vt[s] + drow * VTS + c0);
                u32x2 b = *(const u32x2 *)(Vt[s] + drow * VTS + c1);
                vw[0] = a[0]; vw[1] = a[1]; vw[2] = b[0]; vw[3] = b[1];
                const bf16x8 vf = __builtin_bit_cast(bf16x8, vw);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) o[qb][db] = mfma(vf, pf[qb], o[qb][db]);
            }
        }
    };

#if STAGES == 1
#pragma unroll UNROLL
    for (int kt = 0; kt < n_kt; ++kt) {
        gload(kt);
        swrite(0);
        __syncthreads();
        compute(kt, 0);
        __syncthreads();
    }
#else
    gload(0);
    swrite(0);
    __syncthreads();
#pragma unroll UNROLL
    for (int kt = 0; kt < n_kt; ++kt) {
        if (kt + 1 < n_kt) gload(kt + 1);
        compute(kt, kt & 1);
        if (kt + 1 < n_kt) swrite((kt + 1) & 1);
        __syncthreads();
    }
#endif

#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int q = q0w + qb * MF + lane % MF;
        const float inv = 1.0f / l[qb];
        bf16_t *orow = args.O + base + (size_t)q * AD;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int g = 0; g < ACCN / 4; ++g) {
#if MF == 16
                const int d = db * 16 + 4 * (lane >> 4);
#else
                const int d = db * 32 + g * 8 + 4 * (lane >> 5);
#endif
                u32x2 w;
                w[0] = pack2(o[qb][db][g * 4 + 0] * inv, o[qb][db][g * 4 + 1] * inv);
                w[1] = pack2(o[qb][db][g * 4 + 2] * inv, o[qb][db][g * 4 + 3] * inv);
                *(u32x2 *)(orow + d) = w;
            }
    }
}
