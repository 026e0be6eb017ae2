// bf16 x bf16 -> fp32 MFMA GEMM for gfx950 with fused epilogues.  One
// template serves the gated MLP (dual weight operand + SiLU(g)*u), its down
// projection, the MoE expert GEMMs (gathered / grouped rows) and the
// implicit-GEMM convolution (bias + SiLU).
//
// Compile-time schedule (generated prologue):
//   TM TN TK     workgroup tile (TileSize)
//   WM WN        waves along M and N (Parallel); NT = 64 * WM * WN threads
//   MF           MFMA shape: 16 -> v_mfma_f32_16x16x32_bf16,
//                             32 -> v_mfma_f32_32x32x16_bf16
//   STAGES       1: load, store, compute; 2: LDS double buffer with register
//                prefetch of the next K tile, stored to LDS after the tile's
//                MFMAs; 3: the same, stored half-way through the MFMAs
//                (ComputeLocation); 4: direct-to-LDS loads
//                (global_load_lds_dwordx4) into a ring of three LDS buffers,
//                two K tiles in flight, no register staging (weights stored
//                [N][K], 16-byte vectors, non-im2col rows); 5: as 2 with two
//                register sets, each tile's global loads issued two tiles
//                before its LDS store; 6: ping-pong - eight waves in two
//                groups of four, one wave of each group per SIMD; while one
//                group issues a whole K tile of MFMAs from registers, the
//                other reads its next K tile's fragments from LDS and issues
//                the direct-to-LDS loads of a later tile; the groups swap
//                roles at each barrier (three LDS buffers); 7: a ring of
//                NSTAGE buffers filled by direct-to-LDS buffer loads issued
//                NSTAGE - 1 tiles ahead (range-checked: padded and missing
//                rows load zeros), the next tile's first fragments read
//                during the current tile's last k-step
//   VEC          bf16 elements per global load: 2, 4 or 8 (Vectorize)
//   UNROLL       unroll factor of the K-tile loop (Unroll)
//   LAYOUT       weights stored 0: [K][N], 1: [N][K] (Layout)
//   GRID         0: tile n fastest; 1: tile m fastest, with workgroups
//                regrouped so each XCD owns a contiguous range of tiles;
//                2: tile n fastest, each XCD owning a contiguous range of
//                the tiles that hold rows (for the MoE GEMMs the ones the
//                routing filled), so the workgroups sharing an A tile, and
//                an expert's weights, run on one XCD and its L2
//   NT_FIRST NT_COUNT  column tiles of this launch (default: all of GN)
//   SPLITK       dense rows only: the K range is cut into SPLITK equal parts,
//                one workgroup per (tile, part); part z stores its fp32
//                partial sums (EPI 3; with NB 2 the second operand's to C1)
//                as a compact [SPLITK][GM][launch columns] array, for a
//                separate summing kernel
//   ROWSKIP      MoE only: 1 - a tile past its expert's last row runs a
//                second copy of the main loop that skips the fragment reads
//                and MFMAs of its waves' empty row blocks (ComputeLocation)
//   OCC          waves per SIMD the register allocation must leave room for
//   NB           weight operands sharing the A tile (1, or 2 for gate/up)
//   AMODE        A rows: 0 dense [GM][GK]; 1 MoE gather (row p of expert e
//                reads X[perm[p] / TOPK]); 2 implicit im2col of an NHWC
//                image; 3 MoE grouped dense rows (row p of the permuted
//                hidden matrix)
//   EPI          0 store bf16; 1 + bias, SiLU, store bf16; 2 SiLU(acc0) *
//                acc1, store bf16; 3 store fp32 accumulators (unfused);
//                4 + bias, store bf16 (no activation)
//   GM GN GK     GEMM sizes (GM = rows for AMODE 0/2, total routed rows for
//                AMODE 1/3).  Dense rows (AMODE 0/2) need not fill the last
//                M tile: its missing rows load zeros (register staging) or
//                repeat the tile's first row (direct-to-LDS loads) and are
//                never stored.
//
// LDS holds both operands as rows of TK bf16 (K contiguous).  16-byte
// chunks are XOR-swizzled with the row so that the 16 lanes that share a
// 128-bit LDS access cycle hit distinct banks, for fragment reads and for
// row-major tile writes alike.
//
// The MFMA is issued with the weight fragment as its first operand and the
// activation fragment as its second, so the accumulator holds C^T: each
// lane owns one output row m and runs of 4 consecutive output columns n,
// which the epilogue writes as one 8-byte (bf16) or 16-byte (fp32) store.

#define NT (64 * WM * WN)
#define WTM (TM / WM)
#define WTN (TN / WN)
#define FM (WTM / MF)
#define FN (WTN / MF)
#define CPR (TK / 8)
#define RPL ((16 / CPR) > 0 ? (16 / CPR) : 1)
#ifndef SPLITK
#define SPLITK 1
#endif
#if SPLITK > 1 && (AMODE != 0 || EPI != 3)
#error "a K split needs dense rows and fp32 partial stores"
#endif
// fp32 stores (EPI 3): row stride and first column of the stored block
#if SPLITK > 1
#define OUT_LD (NTN * TN)
#define OUT_C0 (NT_FIRST * TN)
#else
#define OUT_LD GN
#define OUT_C0 0
#endif
#define KTILES (GK / TK / SPLITK)     // K tiles of one workgroup
#define RAGGED_M ((AMODE == 0 || AMODE == 2) && (GM % TM) != 0)
// register-staged vectors per thread (the direct-to-LDS stages do not use
// them; at least 1 keeps their unused arrays well formed)
#define A_LOADS ((TM * TK) / (VEC * NT) > 0 ? (TM * TK) / (VEC * NT) : 1)
#define B_LOADS ((TN * TK) / (VEC * NT) > 0 ? (TN * TK) / (VEC * NT) : 1)
// this launch's column tiles: NT_COUNT tiles starting at tile NT_FIRST (a
// GEMM may be split over two launches by column ranges)
#ifndef NT_FIRST
#define NT_FIRST 0
#endif
#ifndef NT_COUNT
#define NT_COUNT (GN / TN)
#endif
#ifndef ROWSKIP
#define ROWSKIP 0
#endif
#define PART_TILES (ROWSKIP && (AMODE == 1 || AMODE == 3))
#define NTN NT_COUNT

typedef unsigned short bf16_t;

template <int V> struct IntC { static constexpr int value = V; };
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

struct GemmBf16Args {
    const bf16_t *A;
    const bf16_t *B0;
    const bf16_t *B1;
    void *C;
    void *C1;
    const float *bias;
    const int *perm;        // MoE: permuted row -> token * TOPK + slot
    const int *offsets;     // MoE: first permuted row of each expert [NEXP + 1]
    const int *tile_start;  // MoE: first M tile of each expert [NEXP + 1]
};

__device__ __forceinline__ int swz(int row, int chunk) {
    return row * TK + ((chunk ^ ((row / RPL) % CPR)) << 3);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32
__device__ __forceinline__ unsigned pack2(float a, float b) {
    return __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

__device__ __forceinline__ float silu(float x) {
    // x * sigmoid(x); exp(-x) as 2^(-x log2 e) on the hardware exp2 unit.
    return x / (1.0f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
}

__device__ __forceinline__ accT mfma(const bf16x8 &a, const bf16x8 &b, const accT &c) {
#if MF == 16
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
#else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
#endif
}

// Store VEC bf16 held in a register vector into LDS at element offset `off`.
__device__ __forceinline__ void lds_store_vec(bf16_t *lds, int off, const vecT &v) {
    *(vecT *)(lds + off) = v;
}

__device__ __forceinline__ bf16_t vec_elem(const vecT &v, int j) {
#if VEC == 2
    return (bf16_t)(v >> (16 * j));
#else
    return (bf16_t)(v[j >> 1] >> (16 * (j & 1)));
#endif
}

extern "C" __global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
void rc_gemm_bf16(GemmBf16Args args) {
#if STAGES == 4
    // three distinct LDS objects, so the compiler can tell the buffer being
    // filled by direct-to-LDS loads from the one being read
    __shared__ __attribute__((aligned(16))) bf16_t As0[TM * TK], As1[TM * TK], As2[TM * TK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs0[NB][TN * TK], Bs1[NB][TN * TK], Bs2[NB][TN * TK];
#define NBUF 2
    bf16_t (*As)[TM * TK] = nullptr;           // unused with the DMA ring
    bf16_t (*Bs)[NB][TN * TK] = nullptr;
#elif STAGES == 7
    // NSTAGE-deep ring; stage s holds the A tile, then the NB weight tiles
#define STAGE_ELEMS (TM * TK + NB * TN * TK)
    __shared__ __attribute__((aligned(16))) bf16_t ring[NSTAGE * STAGE_ELEMS];
#define NBUF 2
    bf16_t (*As)[TM * TK] = nullptr;           // unused with the ring
    bf16_t (*Bs)[NB][TN * TK] = nullptr;
#elif STAGES == 6
    // three distinct LDS objects per operand (tile t in buffer t % 3)
    __shared__ __attribute__((aligned(16))) bf16_t As0[TM * TK], As1[TM * TK], As2[TM * TK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs0[NB][TN * TK], Bs1[NB][TN * TK], Bs2[NB][TN * TK];
#define NBUF 2
    bf16_t (*As)[TM * TK] = nullptr;           // unused with the ping-pong buffers
    bf16_t (*Bs)[NB][TN * TK] = nullptr;
#else
#define NBUF (STAGES > 1 ? 2 : 1)
    __shared__ __attribute__((aligned(16))) bf16_t As[NBUF][TM * TK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[NBUF][NB][TN * TK];
#endif

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // ---- workgroup -> tile --------------------------------------------
    int bid = blockIdx.x;
    const int nblk = gridDim.x;
#if GRID == 1
    if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
#elif GRID == 2
    // Workgroups reach the 8 XCDs round-robin (workgroup b on XCD b % 8):
    // XCD x takes work items [x * per, (x + 1) * per) of the live ones, in
    // its own dispatch order; the rest of its workgroups exit at once.
#if AMODE == 1 || AMODE == 3
    const int live = args.tile_start[NEXP] * NTN;
#else
    const int live = nblk;
#endif
    if ((nblk & 7) == 0) {
        const int per = (live + 7) >> 3, li = bid >> 3;
        if (li >= per) return;
        bid = (bid & 7) * per + li;
    }
    if (bid >= live) return;
#endif
    // K split: the grid holds SPLITK copies of the tiles, copy z taking K
    // range z; with the XCD regrouping above, an XCD's workgroups fall in
    // one copy (one K range of the operands in its L2)
#if SPLITK > 1
    const int ntiles = nblk / SPLITK;
    const int kz = bid / ntiles;
    bid -= kz * ntiles;
#else
    const int ntiles = nblk;
    constexpr int kz = 0;
#endif
#if GRID == 1
    const int ntm_grid = ntiles / NTN;
    int mt = bid % ntm_grid, nt = bid / ntm_grid;
#else
    (void)ntiles;
    int mt = bid / NTN, nt = bid % NTN;
#endif
    const int n0 = (NT_FIRST + nt) * TN;
    // first K column of this workgroup's range; the operand bases below
    // start there, rows keep their full stride GK
    const size_t KBASE = (size_t)kz * (GK / SPLITK);

#if AMODE == 1 || AMODE == 3
    // Ragged expert groups: find the expert owning M tile `mt`.
    if (mt >= args.tile_start[NEXP]) return;
    int e = 0;
    {
        int lo = 0, hi = NEXP - 1;
        while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if (args.tile_start[mid] <= mt) lo = mid; else hi = mid - 1;
        }
        e = lo;
    }
    const int mrow0 = (mt - args.tile_start[e]) * TM;
    const int row_base = args.offsets[e] + mrow0;                  // first permuted row
    const int rows_valid = min(TM, args.offsets[e + 1] - row_base);
    const size_t wstride = (size_t)GK * GN;
    const bf16_t *B0 = args.B0 + (size_t)e * wstride;
    const bf16_t *const Ab = args.A;
#if NB == 2
    const bf16_t *B1 = args.B1 + (size_t)e * wstride;
#endif
#else
    const int row_base = mt * TM;
    const int rows_valid = RAGGED_M ? min(TM, GM - row_base) : TM;
    const bf16_t *const Ab = args.A + KBASE;
    const bf16_t *B0 = args.B0 + (LAYOUT == 1 ? KBASE : KBASE * GN);
#if NB == 2
    const bf16_t *B1 = args.B1 + (LAYOUT == 1 ? KBASE : KBASE * GN);
#endif
#endif

#if PART_TILES
    // MF-row blocks of this wave that hold routed rows; the products of the
    // blocks past the group's last row would never be stored, so a partial
    // tile skips their fragment reads and MFMAs
    const int fm_live = __builtin_amdgcn_readfirstlane(min(FM, max(0, (rows_valid - wm * WTM + MF - 1) / MF)));
#endif

    // ---- per-thread A row sources (fixed over the K loop) ---------------
    const bf16_t *arow[A_LOADS];
    bool aval[A_LOADS];
#if AMODE == 2
    // Implicit im2col: per load, the element offset of its output pixel's
    // input window corner (filter tap (0, 0), which may lie in the padding)
    // plus its column, and a mask of the filter taps that fall inside the
    // image; a K tile then only adds the tap's offset (wave-uniform).
    long long a_off[A_LOADS];
    unsigned a_mask[A_LOADS];
#endif
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
        int v = tid + i * NT;
        int r = v / (TK / VEC);
#if AMODE == 1 || AMODE == 3
        aval[i] = r < rows_valid;
#else
        aval[i] = !RAGGED_M || r < rows_valid;
#endif
#if AMODE == 0
        arow[i] = Ab + (size_t)(aval[i] ? row_base + r : 0) * GK;
#elif AMODE == 1
        int tok = aval[i] ? args.perm[row_base + r] / TOPK : 0;
        arow[i] = Ab + (size_t)tok * GK;
#elif AMODE == 3
        arow[i] = Ab + (size_t)(aval[i] ? row_base + r : 0) * GK;
#else
        const int m = row_base + r, c = (v % (TK / VEC)) * VEC;
        const int n = m / (CV_P * CV_Q), p = (m / CV_Q) % CV_P, q = m % CV_Q;
        a_off[i] = ((long long)(n * CV_H + p - CV_PAD) * CV_W + (q - CV_PAD)) * CV_C + c;
        unsigned mask = 0;
#pragma unroll
        for (int tap = 0; tap < GK / CV_C; ++tap) {
            const int ih = p + tap / CV_S - CV_PAD, iw = q + tap % CV_S - CV_PAD;
            if (ih >= 0 && ih < CV_H && iw >= 0 && iw < CV_W) mask |= 1u << tap;
        }
        a_mask[i] = aval[i] ? mask : 0u;      // rows past GM load nothing
        arow[i] = Ab;
#endif
    }

    accT acc[NB][FM][FN];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) acc[b][i][j][r] = 0.f;

    // register staging sets: tile t uses set t % NSET
#define NSET (STAGES == 5 ? 2 : 1)
    vecT ra[NSET][A_LOADS];
    vecT rb[NSET][NB][B_LOADS];

    auto gload = [&](int k0, int set) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            int v = tid + i * NT;
            int c = (v % (TK / VEC)) * VEC;
#if AMODE == 2
            // K tile k0 lies in filter tap (r, s) = divmod(k0 / C, S), channels
            // k0 % C ..; the offsets below are the same for the whole wave.
            (void)c;
            const int tap = k0 / CV_C;
            const long long tap_off = ((long long)(tap / CV_S) * CV_W + tap % CV_S) * CV_C + (k0 - tap * CV_C);
            ra[set][i] = ((a_mask[i] >> tap) & 1u) ? *(const vecT *)(Ab + (a_off[i] + tap_off)) : (vecT)0;
#else
            ra[set][i] = aval[i] ? *(const vecT *)(arow[i] + k0 + c) : (vecT)0;
#endif
        }
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            int v = tid + i * NT;
#if LAYOUT == 1
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
            size_t off = (size_t)(n0 + r) * GK + k0 + c;
#else
            int r = v / (TN / VEC), c = (v % (TN / VEC)) * VEC;
            size_t off = (size_t)(k0 + r) * GN + n0 + c;
#endif
            rb[set][0][i] = *(const vecT *)(B0 + off);
#if NB == 2
            rb[set][1][i] = *(const vecT *)(B1 + off);
#endif
        }
    };

    auto swrite = [&](int s, int set) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            int v = tid + i * NT;
            int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
            lds_store_vec(As[s], swz(r, c >> 3) + (c & 7), ra[set][i]);
        }
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int i = 0; i < B_LOADS; ++i) {
                int v = tid + i * NT;
#if LAYOUT == 1
                int r = v / (TK / VEC), c = (v % (TK / VEC)) * VEC;
                lds_store_vec(Bs[s][b], swz(r, c >> 3) + (c & 7), rb[set][b][i]);
#else
                int kr = v / (TN / VEC), c = (v % (TN / VEC)) * VEC;
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    Bs[s][b][swz(c + j, kr >> 3) + (kr & 7)] = vec_elem(rb[set][b][i], j);
#endif
            }
    };

    // Fragments of one k-step: FM activation and NB x FN weight fragments.
    struct Frags {
        bf16x8 a[FM];
        bf16x8 b[NB][FN];
    };
    // The swizzle's XOR depends on the row modulo MF only (MF / RPL is a
    // multiple of CPR for every legal tile_k), so each lane's fragment
    // offset within an MF-row block is computed once per k-step and every
    // block adds a constant.
    int foff[TK / KSTEP];
#pragma unroll
    for (int ks = 0; ks < TK / KSTEP; ++ks) foff[ks] = swz(lane % MF, ks * (KSTEP / 8) + lane / MF);
    // `part` (IntC<0> or IntC<1>) selects the full tile or a partial MoE
    // tile whose wave holds fm_live live row blocks.
    auto load_frags = [&](const bf16_t *la, const bf16_t (*lb)[TN * TK], int ks, Frags &f, auto part) {
#if PART_TILES
        if constexpr (decltype(part)::value)
            if (fm_live == 0) return;
#endif
#pragma unroll
        for (int i = 0; i < FM; ++i)
            f.a[i] = *(const bf16x8 *)(la + (wm * WTM + i * MF) * TK + foff[ks]);
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                f.b[b][j] = *(const bf16x8 *)(lb[b] + (wn * WTN + j * MF) * TK + foff[ks]);
    };
    auto mfmas = [&](const Frags &f, auto part) {
        if constexpr (decltype(part)::value) {
#if PART_TILES
#pragma unroll
            for (int i = 0; i < FM; ++i)
                if (i < fm_live) {
#pragma unroll
                    for (int b = 0; b < NB; ++b)
#pragma unroll
                        for (int j = 0; j < FN; ++j) acc[b][i][j] = mfma(f.b[b][j], f.a[i], acc[b][i][j]);
                }
#endif
        } else {
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j) acc[b][i][j] = mfma(f.b[b][j], f.a[i], acc[b][i][j]);
        }
    };
    // Runs a main loop `run(part)`: a second copy for partial MoE tiles.
    auto run_tiles = [&](auto &&run) {
#if PART_TILES
        if (fm_live == FM) run(IntC<0>{});
        else run(IntC<1>{});
#else
        run(IntC<0>{});
#endif
    };
    // One K tile from LDS buffer s.  The fragments of k-step ks + 1 are read
    // while the MFMAs of k-step ks issue; `mid` (the LDS store of the next
    // tile into the other buffer) runs halfway through the MFMAs.
    auto compute_at = [&](const bf16_t *la, const bf16_t (*lb)[TN * TK], auto &&mid, auto part) {
        constexpr int KS = TK / KSTEP;
        Frags f[2];
        load_frags(la, lb, 0, f[0], part);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS) load_frags(la, lb, ks + 1, f[(ks + 1) & 1], part);
            if (ks == KS / 2) mid();
            mfmas(f[ks & 1], part);
        }
        if (KS == 1) mid();
    };
    auto compute = [&](int s, auto &&mid, auto part) { compute_at(As[s], Bs[s], mid, part); };

    auto nothing = [] {};
#if STAGES == 4
    // Direct-to-LDS loads: one global_load_lds_dwordx4 moves 64 lanes x 16 B
    // into 1 KiB of LDS at a wave-uniform base, lane i at byte 16 i.  The
    // swizzle is applied by choosing which global chunk each lane fetches:
    // LDS chunk c of the tile holds row c / CPR, logical chunk
    // (c % CPR) ^ ((row / RPL) % CPR) of that row (the XOR is an involution).
    typedef __attribute__((address_space(3))) void *lds_vp;
    typedef __attribute__((address_space(1))) void *gbl_vp;
    constexpr int NWV = WM * WN;
    constexpr int A_WL = TM * TK / 8 / 64 / NWV;     // wave-loads per wave, A tile
    constexpr int B_WL = TN * TK / 8 / 64 / NWV;     // per weight operand
    constexpr int LPT = A_WL + NB * B_WL;            // loads per lane per K tile
    const bf16_t *a_src[A_WL];
    const bf16_t *b_src[NB][B_WL];
#pragma unroll
    for (int j = 0; j < A_WL; ++j) {
        const int c = (wave * A_WL + j) * 64 + lane;
        const int row = c / CPR, lc = (c % CPR) ^ ((row / RPL) % CPR);
#if AMODE == 0
        // rows past GM read the tile's first row; their products are never stored
        a_src[j] = Ab + (size_t)(row_base + (RAGGED_M && row >= rows_valid ? 0 : row)) * GK + lc * 8;
#elif AMODE == 1
        // rows past the group read a valid row; their products are never stored
        const int tok = args.perm[row_base + (row < rows_valid ? row : 0)] / TOPK;
        a_src[j] = Ab + (size_t)tok * GK + lc * 8;
#else
        a_src[j] = Ab + (size_t)(row_base + (row < rows_valid ? row : 0)) * GK + lc * 8;
#endif
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < B_WL; ++j) {
            const int c = (wave * B_WL + j) * 64 + lane;
            const int row = c / CPR, lc = (c % CPR) ^ ((row / RPL) % CPR);
            b_src[b][j] = (b == 0 ? B0 :
#if NB == 2
                           B1
#else
                           B0
#endif
                           ) + (size_t)(n0 + row) * GK + lc * 8;
        }
    auto gload_lds = [&](int k0, bf16_t *la, bf16_t (*lb)[TN * TK]) {
#pragma unroll
        for (int j = 0; j < A_WL; ++j)
            __builtin_amdgcn_global_load_lds((gbl_vp)(a_src[j] + k0),
                                             (lds_vp)(la + (wave * A_WL + j) * 512), 16, 0, 0);
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int j = 0; j < B_WL; ++j)
                __builtin_amdgcn_global_load_lds((gbl_vp)(b_src[b][j] + k0),
                                                 (lds_vp)(lb[b] + (wave * B_WL + j) * 512), 16, 0, 0);
    };
    // s_waitcnt with only the vector-memory count constrained (expcnt and
    // lgkmcnt at their maxima): at most n loads of this wave still in flight
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    gload_lds(0, As0, Bs0);
    if (KTILES > 1) {
        gload_lds(TK, As1, Bs1);
        WAIT_VM(LPT);
    } else {
        WAIT_VM(0);
    }
    __syncthreads();
    // tile kt sits in buffer kt % 3; buffer (kt + 2) % 3 held tile kt - 1,
    // finished before the last barrier, and receives tile kt + 2
    auto body = [&](int kt, bf16_t *cur_a, bf16_t (*cur_b)[TN * TK], bf16_t *fill_a,
                    bf16_t (*fill_b)[TN * TK], auto part) {
        if (kt + 2 < KTILES) gload_lds((kt + 2) * TK, fill_a, fill_b);
        compute_at(cur_a, cur_b, nothing, part);
        if (kt + 2 < KTILES) {
            WAIT_VM(LPT);          // tile kt + 1 has landed; tile kt + 2 may be in flight
        } else {
            WAIT_VM(0);
        }
        // Barrier without a release fence: __syncthreads() would also wait for
        // tile kt + 2's loads.  LDS written by this wave's completed loads is
        // visible to the workgroup once the barrier is passed; the memory
        // clobber keeps the compiler from moving LDS accesses across it.
        __builtin_amdgcn_s_waitcnt(0xC07F);      // lgkmcnt(0): this wave's LDS reads are done
        asm volatile("s_barrier" ::: "memory");
    };
    run_tiles([&](auto part) __attribute__((always_inline)) {
        for (int kt = 0; kt < KTILES; kt += 3) {
            body(kt, As0, Bs0, As2, Bs2, part);
            if (kt + 1 < KTILES) body(kt + 1, As1, Bs1, As0, Bs0, part);
            if (kt + 2 < KTILES) body(kt + 2, As2, Bs2, As1, Bs1, part);
        }
    });
#undef WAIT_VM
#elif STAGES == 7
    // Deep direct-to-LDS ring.  buffer_load_dwordx4 ... lds moves 64 lanes x
    // 16 B into 1 KiB of LDS at a wave-uniform base (M0); the swizzle is
    // applied by choosing which global chunk each lane fetches, as for
    // stages 4.  The loads go through buffer resources whose range checking
    // returns zeros for an offset past the buffer: rows past the operator's
    // rows and taps of an im2col window that fall in the padding get offset
    // OOB and load zeros.  Tile t goes to stage t % NSTAGE and is issued
    // NSTAGE - 1 tiles ahead; the fragments of tile t + 1's first k-step are
    // read during tile t's last k-step, so each tile starts its MFMAs at
    // once after the one barrier per tile (which also frees the stage of
    // tile t - 1 for tile t + NSTAGE - 1).  The loads are inline assembly,
    // invisible to the compiler's wait-count bookkeeping; the waits below
    // order the ring (loads complete in order).
    typedef int i32x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) bf16_t *lds_p;
    constexpr int NWV = WM * WN;
    constexpr int A_WL = TM * TK / 512 / NWV;        // wave-loads per wave, A tile
    constexpr int B_WL = TN * TK / 512 / NWV;        // per weight operand
    constexpr int LPT = A_WL + NB * B_WL;            // loads per lane per tile
    constexpr int KS = TK / KSTEP;
    constexpr unsigned OOB = 0x80000000u;            // past every operand: loads zeros
    auto rsrc = [](const void *base, unsigned long long bytes) {
        const unsigned long long a = (unsigned long long)base;
        i32x4 r;
        r[0] = __builtin_amdgcn_readfirstlane((int)(unsigned)a);
        r[1] = __builtin_amdgcn_readfirstlane((int)((unsigned)(a >> 32) & 0xFFFFu));   // stride 0
        r[2] = __builtin_amdgcn_readfirstlane((int)(unsigned)(bytes < 0xFFFFFFFFull ? bytes : 0xFFFFFFFFull));
        r[3] = 0x00020000;                                                             // raw dword access
        return r;
    };
#if AMODE == 1
    const i32x4 rsA = rsrc(Ab, (unsigned long long)(GM / TOPK) * GK * 2);
#elif AMODE == 2
    const i32x4 rsA = rsrc(Ab, (unsigned long long)(GM / (CV_P * CV_Q)) * CV_H * CV_W * CV_C * 2);
#else
    const i32x4 rsA = rsrc(Ab, ((unsigned long long)GM * GK - KBASE) * 2);
#endif
    i32x4 rsB[NB];
    rsB[0] = rsrc(B0, ((unsigned long long)GN * GK - KBASE) * 2);
#if NB == 2
    rsB[1] = rsrc(B1, ((unsigned long long)GN * GK - KBASE) * 2);
#endif
    // per-lane byte offsets of each wave-load at k0 = 0
    unsigned a_off7[A_WL];
    bool a_ok7[A_WL];
#if AMODE == 2
    int a_cor7[A_WL];                                 // window corner (may lie in the padding), bytes
    unsigned a_msk7[A_WL];
#endif
#pragma unroll
    for (int j = 0; j < A_WL; ++j) {
        const int c = (wave * A_WL + j) * 64 + lane;
        const int row = c / CPR, lc = (c % CPR) ^ ((row / RPL) % CPR);
#if AMODE == 0 || AMODE == 3
        a_ok7[j] = row < rows_valid;
        a_off7[j] = (unsigned)(((size_t)(row_base + row) * GK + lc * 8) * 2);
#elif AMODE == 1
        a_ok7[j] = row < rows_valid;
        const int tok = args.perm[row_base + (a_ok7[j] ? row : 0)] / TOPK;
        a_off7[j] = (unsigned)(((size_t)tok * GK + lc * 8) * 2);
#else
        const int m = row_base + row;
        a_ok7[j] = m < GM;
        const int n = m / (CV_P * CV_Q), p = (m / CV_Q) % CV_P, q = m % CV_Q;
        a_cor7[j] = 2 * (((n * CV_H + p - CV_PAD) * CV_W + (q - CV_PAD)) * CV_C + lc * 8);
        unsigned mask = 0;
#pragma unroll
        for (int tap = 0; tap < GK / CV_C; ++tap) {
            const int ih = p + tap / CV_S - CV_PAD, iw = q + tap % CV_S - CV_PAD;
            if (ih >= 0 && ih < CV_H && iw >= 0 && iw < CV_W) mask |= 1u << tap;
        }
        a_msk7[j] = a_ok7[j] ? mask : 0u;
        a_off7[j] = 0;
#endif
    }
    unsigned b_off7[B_WL];
#pragma unroll
    for (int j = 0; j < B_WL; ++j) {
        const int c = (wave * B_WL + j) * 64 + lane;
        const int row = c / CPR, lc = (c % CPR) ^ ((row / RPL) % CPR);
        b_off7[j] = (unsigned)(((size_t)(n0 + row) * GK + lc * 8) * 2);
    }
    auto dma = [&](unsigned off, const i32x4 &rs, unsigned lds_addr) {
        asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                     :: "v"(off), "s"(rs), "s"(lds_addr) : "memory", "m0");
    };
    const unsigned ring0 = (unsigned)(size_t)(lds_p)ring;
    const int wv = __builtin_amdgcn_readfirstlane(wave);      // wave-uniform, in a scalar register
    auto issue = [&](int kt, int st) {
        const int k0 = kt * TK;
        const unsigned sb = ring0 + (unsigned)(st * STAGE_ELEMS * 2);
#if AMODE == 2
        const int tap = k0 / CV_C;
        const int tap_off = 2 * (((tap / CV_S) * CV_W + tap % CV_S) * CV_C + (k0 - tap * CV_C));
#endif
#pragma unroll
        for (int j = 0; j < A_WL; ++j) {
#if AMODE == 2
            const unsigned off = ((a_msk7[j] >> tap) & 1u) ? (unsigned)(a_cor7[j] + tap_off) : OOB;
#else
            const unsigned off = a_ok7[j] ? a_off7[j] + 2u * k0 : OOB;
#endif
            dma(off, rsA, sb + (unsigned)((wv * A_WL + j) * 1024));
        }
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int j = 0; j < B_WL; ++j)
                dma(b_off7[j] + 2u * k0, rsB[b],
                    sb + (unsigned)(TM * TK * 2 + b * TN * TK * 2 + (wv * B_WL + j) * 1024));
    };
    // s_waitcnt with only the vector-memory count constrained
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    // wait until at most `newer` tiles' loads of this wave are in flight
    auto wait_tiles = [&](int newer) {
        switch (newer) {
            case 1: WAIT_VM(LPT); break;
#if NSTAGE > 3
            case 2: WAIT_VM(2 * LPT); break;
#endif
#if NSTAGE > 4
            case 3: WAIT_VM(3 * LPT); break;
#endif
#if NSTAGE > 5
            case 4: WAIT_VM(4 * LPT); break;
#endif
#if NSTAGE > 6
            case 5: WAIT_VM(5 * LPT); break;
#endif
#if NSTAGE > 7
            case 6: WAIT_VM(6 * LPT); break;
#endif
#if NSTAGE > 8
            case 7: WAIT_VM(7 * LPT); break;
#endif
#if NSTAGE > 9
            case 8: WAIT_VM(8 * LPT); break;
#endif
#if NSTAGE > 10
            case 9: WAIT_VM(9 * LPT); break;
#endif
#if NSTAGE > 11
            case 10: WAIT_VM(10 * LPT); break;
#endif
            default: WAIT_VM(0); break;
        }
    };
    auto stage_a = [&](int t) { return (const bf16_t *)(ring + (t % NSTAGE) * STAGE_ELEMS); };
    auto stage_b = [&](const bf16_t *la) { return (const bf16_t (*)[TN * TK])(la + TM * TK); };
    // MFMAs of one k-step interleaved with the next k-step's fragment reads
    constexpr int NMF = NB * FM * FN, NRD = FM + NB * FN;
    auto kstep = [&](const Frags &cur, const bf16_t *ln, int ksn, Frags &nxt, auto part) {
        load_frags(ln, stage_b(ln), ksn, nxt, part);
        mfmas(cur, part);
        if constexpr (!decltype(part)::value) {
#pragma unroll
            for (int r = 0; r < NRD; ++r) {
                __builtin_amdgcn_sched_group_barrier(0x008, NMF / NRD > 0 ? NMF / NRD : 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, NMF, 0);
        }
    };
    Frags f7[2];
#pragma unroll
    for (int u = 0; u < NSTAGE - 1; ++u)
        if (u < KTILES) issue(u, u);
    wait_tiles(min(NSTAGE - 2, KTILES - 1));
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("s_barrier" ::: "memory");
    auto body7 = [&](int t, auto par, auto part) {
        constexpr int P = decltype(par)::value;
        if (t + 1 < KTILES) {
            // tile t + 1 has landed; every wave is done with tile t - 1's stage
            wait_tiles(min(KTILES - 1, t + NSTAGE - 2) - (t + 1));
            __builtin_amdgcn_s_waitcnt(0xC07F);
            asm volatile("s_barrier" ::: "memory");
            if (t + NSTAGE - 1 < KTILES) issue(t + NSTAGE - 1, (t + NSTAGE - 1) % NSTAGE);
        }
        const bf16_t *la = stage_a(t);
        const bf16_t *ln = stage_a(t + 1);   // the last tile reads a stale stage; unused
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int ci = (P * KS + ks) & 1;          // a constant once unrolled
            if (ks + 1 < KS) {
                if (ci == 0) kstep(f7[0], la, ks + 1, f7[1], part);
                else kstep(f7[1], la, ks + 1, f7[0], part);
            } else {
                if (ci == 0) kstep(f7[0], ln, 0, f7[1], part);
                else kstep(f7[1], ln, 0, f7[0], part);
            }
        }
    };
    run_tiles([&](auto part) __attribute__((always_inline)) {
        load_frags(stage_a(0), stage_b(stage_a(0)), 0, f7[0], part);
        for (int t = 0; t < KTILES; t += 2) {
            body7(t, IntC<0>{}, part);
            if (t + 1 < KTILES) body7(t + 1, IntC<1>{}, part);
        }
    });
#undef WAIT_VM
#elif STAGES == 6
    // Ping-pong.  Waves 0-3 (group 0) and 4-7 (group 1) hold one wave per
    // SIMD each.  Time is cut into slots separated by workgroup barriers:
    //   slot 2t:     group 0 computes K tile t from registers;
    //                group 1 reads tile t's fragments (LDS buffer t % 3)
    //   slot 2t + 1: group 0 reads tile t + 1's fragments and loads tile
    //                t + 3 into buffer t % 3 (direct to LDS);
    //                group 1 computes tile t
    // so on every SIMD one wave issues MFMAs while the other moves data.
    // Buffer t % 3 was last read by group 1 in slot 2t, before the barrier
    // that opens slot 2t + 1; tile t + 3's loads have the slots up to group
    // 0's read in slot 2t + 5 to land (waited for at the end of slot 2t + 4,
    // with the next tile's loads still in flight).  Group 0 issues all
    // direct-to-LDS loads.
    typedef __attribute__((address_space(3))) void *lds_vp;
    typedef __attribute__((address_space(1))) void *gbl_vp;
    constexpr int A_WL = TM * TK / 8 / 64 / 4;       // wave-loads per loading wave, A tile
    constexpr int B_WL = TN * TK / 8 / 64 / 4;       // per weight operand
    const int grp = __builtin_amdgcn_readfirstlane(wave >> 2);
    const int lw = __builtin_amdgcn_readfirstlane(wave & 3);
    // Source of the 16-byte chunk a lane moves in wave-load W of a tile: row
    // W * (64 / CPR) + lane / CPR, chunk lc0 ^ 4 x with lc0 = (lane % CPR) ^
    // (lane / CPR / RPL) and x = W % (CPR / 4) (the row swizzle of load W
    // differs from load 0 by a wave-uniform XOR).  So a lane needs one byte
    // offset per distinct x for dense rows; the rest of each address is
    // wave-uniform and lives in scalar registers.
    constexpr int NX = CPR / 4;
    const int r_l = lane / CPR;
    const int lc0 = (lane % CPR) ^ (r_l / RPL);
    unsigned voff[NX];
#pragma unroll
    for (int x = 0; x < NX; ++x) voff[x] = (unsigned)(r_l * GK * 2 + ((lc0 ^ (4 * x)) << 4));
#if AMODE != 0 || RAGGED_M
    // gathered or ragged rows: one offset (from the A base) per load
    unsigned a_off[A_WL];
#pragma unroll
    for (int j = 0; j < A_WL; ++j) {
        const int row = (lw * A_WL + j) * (64 / CPR) + r_l;
        const int lc = lc0 ^ (4 * ((lw * A_WL + j) % NX));
#if AMODE == 1
        // rows past the group read a valid row; their products are never stored
        const int tok = args.perm[row_base + (row < rows_valid ? row : 0)] / TOPK;
        a_off[j] = (unsigned)(tok * GK * 2 + (lc << 4));
#else
        a_off[j] = (unsigned)((row_base + (row < rows_valid ? row : 0)) * GK * 2 + (lc << 4));
#endif
    }
#endif
    auto gload_lds = [&](int k0, bf16_t *la, bf16_t (*lb)[TN * TK]) {
        // the empty asm keeps each address a scalar base + this lane offset
        // (no per-load 64-bit address registers hoisted out of the loop)
        unsigned vo[NX];
#pragma unroll
        for (int x = 0; x < NX; ++x) {
            vo[x] = voff[x];
            asm volatile("" : "+v"(vo[x]));
        }
#if AMODE != 0 || RAGGED_M
        unsigned ao[A_WL];
#pragma unroll
        for (int j = 0; j < A_WL; ++j) {
            ao[j] = a_off[j];
            asm volatile("" : "+v"(ao[j]));
        }
#endif
#pragma unroll
        for (int j = 0; j < A_WL; ++j) {
            const int W = lw * A_WL + j;
#if AMODE == 0 && !RAGGED_M
            const char *base = (const char *)(Ab + ((size_t)row_base + W * (64 / CPR)) * GK + k0);
            __builtin_amdgcn_global_load_lds((gbl_vp)(base + vo[A_WL % NX == 0 ? j % NX : W % NX]), (lds_vp)(la + W * 512), 16, 0, 0);
#else
            const char *base = (const char *)(Ab + k0);
            __builtin_amdgcn_global_load_lds((gbl_vp)(base + ao[j]), (lds_vp)(la + W * 512), 16, 0, 0);
#endif
        }
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int j = 0; j < B_WL; ++j) {
                const int W = lw * B_WL + j;
                const bf16_t *bb = b == 0 ? B0 :
#if NB == 2
                                   B1;
#else
                                   B0;
#endif
                const char *base = (const char *)(bb + ((size_t)n0 + W * (64 / CPR)) * GK + k0);
                __builtin_amdgcn_global_load_lds((gbl_vp)(base + vo[B_WL % NX == 0 ? j % NX : W % NX]), (lds_vp)(lb[b] + W * 512), 16, 0, 0);
            }
    };
#define WAIT_VM0() __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8))
#define WAIT_LGKM0() __builtin_amdgcn_s_waitcnt(0xC07F)
    // barrier without a release fence (which would also wait for in-flight
    // direct-to-LDS loads); the clobber keeps LDS accesses on their side
#define SLOT_BARRIER() asm volatile("s_barrier" ::: "memory")
    Frags fr[TK / KSTEP];
    // One LDS base address per operand and k-step, computed where it is used
    // (the empty asm keeps the compiler from hoisting one address register
    // per fragment out of the loop); fragments are base + immediate offset.
    typedef __attribute__((address_space(3))) const bf16x8 *lfp;
    auto read_tile = [&](const bf16_t *la, const bf16_t (*lb)[TN * TK]) {
#pragma unroll
        for (int ks = 0; ks < TK / KSTEP; ++ks) {
            lfp pa = (lfp)(la + wm * WTM * TK + foff[ks]);
            asm volatile("" : "+v"(pa));
#pragma unroll
            for (int i = 0; i < FM; ++i) fr[ks].a[i] = pa[i * MF * TK / 8];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                lfp pb = (lfp)(lb[b] + wn * WTN * TK + foff[ks]);
                asm volatile("" : "+v"(pb));
#pragma unroll
                for (int j = 0; j < FN; ++j) fr[ks].b[b][j] = pb[j * MF * TK / 8];
            }
        }
        WAIT_LGKM0();
    };
    auto compute_tile = [&]() {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int ks = 0; ks < TK / KSTEP; ++ks) mfmas(fr[ks], IntC<0>{});
        __builtin_amdgcn_s_setprio(0);
    };
    // Both groups run the same loop, "compute tile t; barrier; memory work
    // for tile t + 1; barrier", group 1 entering it one slot later (after
    // reading tile 0 while group 0 computes it) and group 0 leaving with one
    // extra barrier, so the MFMAs have a single site and the accumulators
    // stay in place.
    constexpr int LPT = A_WL + NB * B_WL;           // loads per loading wave per tile
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    if (grp == 0) {
        gload_lds(0, As0, Bs0);
        if (KTILES > 1) gload_lds(TK, As1, Bs1);
        if (KTILES > 2) gload_lds(2 * TK, As2, Bs2);
        if (KTILES > 2) {
            WAIT_VM(LPT);          // tiles 0 and 1 have landed
        } else {
            WAIT_VM0();
        }
    }
    SLOT_BARRIER();
    if (grp == 0) read_tile(As0, Bs0);
    SLOT_BARRIER();
    if (grp == 1) {
        read_tile(As0, Bs0);       // slot 0, while group 0 computes tile 0
        SLOT_BARRIER();
    }
    // tile t sits in buffer cur, t + 1 in nxt; tile t + 3 goes to cur
    auto step = [&](int t, bf16_t *cur_a, bf16_t (*cur_b)[TN * TK], bf16_t *nxt_a,
                    bf16_t (*nxt_b)[TN * TK]) {
        compute_tile();
        if (grp == 0) {
            // tile t + 1 has landed (tile t + 2 may still be in flight)
            if (t + 2 < KTILES) {
                WAIT_VM(LPT);
            } else {
                WAIT_VM0();
            }
        }
        SLOT_BARRIER();
        if (t + 1 < KTILES) {
            if (grp == 0) {
                if (t + 3 < KTILES) gload_lds((t + 3) * TK, cur_a, cur_b);
                read_tile(nxt_a, nxt_b);
            } else {
                read_tile(nxt_a, nxt_b);
            }
        }
        SLOT_BARRIER();
    };
    for (int t = 0; t < KTILES; t += 3) {
        step(t, As0, Bs0, As1, Bs1);
        if (t + 1 < KTILES) step(t + 1, As1, Bs1, As2, Bs2);
        if (t + 2 < KTILES) step(t + 2, As2, Bs2, As0, Bs0);
    }
    if (grp == 0) SLOT_BARRIER();
#undef WAIT_VM
#undef WAIT_VM0
#undef WAIT_LGKM0
#undef SLOT_BARRIER
#elif STAGES == 1
    run_tiles([&](auto part) __attribute__((always_inline)) {
#pragma unroll UNROLL
        for (int kt = 0; kt < KTILES; ++kt) {
            gload(kt * TK, 0);
            swrite(0, 0);
            __syncthreads();
            compute(0, nothing, part);
            __syncthreads();
        }
    });
#elif STAGES == 5
    // Tile t lives in register set t % 2 and LDS buffer t % 2.  Its loads are
    // issued at the end of iteration t - 3 (right after the set's previous
    // tile was stored) and it is stored at the end of iteration t - 1, so two
    // tiles of MFMAs cover the load latency.  The loop is unrolled by two so
    // that every set and buffer index is a constant.
    gload(0, 0);
    swrite(0, 0);
    if (KTILES > 1) gload(TK, 1);
    if (KTILES > 2) gload(2 * TK, 0);
    __syncthreads();
    auto body = [&](int kt, auto par, auto part) {
        constexpr int P = decltype(par)::value;
        compute(P, nothing, part);
        if (kt + 1 < KTILES) swrite(1 - P, 1 - P);
        __syncthreads();
        if (kt + 3 < KTILES) gload((kt + 3) * TK, 1 - P);
    };
    run_tiles([&](auto part) __attribute__((always_inline)) {
        for (int kt = 0; kt < KTILES; kt += 2) {
            body(kt, IntC<0>{}, part);
            if (kt + 1 < KTILES) body(kt + 1, IntC<1>{}, part);
        }
    });
#else
    gload(0, 0);
    swrite(0, 0);
    __syncthreads();
    run_tiles([&](auto part) __attribute__((always_inline)) {
#pragma unroll UNROLL
        for (int kt = 0; kt < KTILES; ++kt) {
            // buffer (kt + 1) & 1 was last read in iteration kt - 1, which ended
            // with a barrier, so it may be overwritten during this tile's MFMAs
            if (kt + 1 < KTILES) gload((kt + 1) * TK, 0);
            const int nxt = (kt + 1) & 1;
            const bool more = kt + 1 < KTILES;
#if STAGES == 3
            compute(kt & 1, [&] {
                if (more) swrite(nxt, 0);
            }, part);
#else
            compute(kt & 1, nothing, part);
            if (more) swrite(nxt, 0);
#endif
            __syncthreads();
        }
    });
#endif

    // ---- epilogue --------------------------------------------------------
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int mloc = wm * WTM + i * MF + lane % MF;
        if (mloc >= rows_valid) continue;
        const size_t orow = (size_t)(row_base + mloc) * GN;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int g = 0; g < ACCN / 4; ++g) {
                // columns n .. n+3 of this lane's row
#if MF == 16
                const int n = n0 + wn * WTN + j * MF + 4 * (lane >> 4);
#else
                const int n = n0 + wn * WTN + j * MF + g * 8 + 4 * (lane >> 5);
#endif
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = acc[0][i][j][g * 4 + r];
#if EPI == 3
                const size_t po = (size_t)kz * GM * OUT_LD + (size_t)(row_base + mloc) * OUT_LD + (n - OUT_C0);
                *(f32x4 *)((float *)args.C + po) = f32x4{v[0], v[1], v[2], v[3]};
#if NB == 2
                *(f32x4 *)((float *)args.C1 + po) =
                    f32x4{acc[1][i][j][g * 4 + 0], acc[1][i][j][g * 4 + 1], acc[1][i][j][g * 4 + 2],
                          acc[1][i][j][g * 4 + 3]};
#endif
#else
#if EPI == 1
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = silu(v[r] + args.bias[n + r]);
#elif EPI == 2
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = silu(v[r]) * acc[1][i][j][g * 4 + r];
#elif EPI == 4
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = v[r] + args.bias[n + r];
#endif
                u32x2 packed;
                packed[0] = pack2(v[0], v[1]);
                packed[1] = pack2(v[2], v[3]);
                *(u32x2 *)((bf16_t *)args.C + orow + n) = packed;
#endif
            }
        }
    }
}
