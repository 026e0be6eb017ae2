// Softmax attention forward for gfx950, bf16 Q/K/V/O [B][H][S][D], fp32
// scores, online (blockwise) softmax, bf16 MFMA for both products.
//
// Compile-time schedule (generated prologue):
//   BM           query rows per workgroup (TileSize)
//   BN           keys per tile (TileSize)
//   NW           wave row groups; each owns BM / NW query rows (Parallel)
//   SPLITS       key splits inside the workgroup (Parallel): NW * SPLITS
//                waves; split s takes key tiles s, s + SPLITS, ... with its
//                own online-softmax state, and the states of the splits are
//                merged through LDS at the end (exact: partial outputs and
//                sums relative to their own maxima are rescaled to the joint
//                maximum)
//   MF           MFMA shape 16 (16x16x32) or 32 (32x32x16)
//   STAGES       1: load tile, compute; 2: double-buffered K/V tiles with
//                register prefetch of the next tile; 3: as 2, plus the
//                scores of the next tile computed ahead of this tile's
//                softmax (software pipeline); 4: direct global-to-LDS loads
//                into a ring of three K/V buffers, two tiles in flight
//                while one is computed, V kept key-major and read with the
//                transposing LDS load; 5: as 4 with a ring of four slots
//                per key split and the scores of the split's next tile
//                computed ahead of this tile's softmax (ComputeLocation)
//   VEC          bf16 per global load of K (Vectorize)
//   UNROLL       unroll factor of the key-tile loop (Unroll)
//   ORDER        0: query tiles in order; 1: longest (last) query tiles
//                first; 2: paired - workgroup b and b + half take query
//                tiles t and NQT-1-t, so that co-resident pairs carry equal
//                causal work
//   OCC          waves per SIMD the register allocation must leave room for
//   CHUNK        0: a workgroup runs a query tile's whole key range; n > 0:
//                the key range is cut into work items of at most n key tiles
//                (Parallel).  Items of a cut tile leave their unnormalised
//                state (O, m, l) in the workspace and rc_attention_combine
//                merges them, which shortens the longest workgroup's chain
//                of dependent key tiles
//   AB AH AS AD  batch, heads, sequence length, head dim.  AS need not be a
//                multiple of BM or BN: the last query tile's rows past AS
//                read row AS - 1 of Q and are not stored; the last key
//                tile's rows past AS load zeros (register staging) or
//                repeat row AS - 1 (direct-to-LDS loads), and their scores
//                are masked (the causal mask already hides them from every
//                stored query)
//   CAUSAL       top-left aligned causal mask (key j visible iff j <= i)
//   SCALE_LOG2   log2(e) / sqrt(AD): scores are kept in log2 units
//
// Layout of the products.  Scores are computed transposed, S^T = K Q^T,
// with K as the first MFMA operand: each lane then holds the scores of ONE
// query (column lane % MF) for several keys, so the softmax statistics
// (running max m and sum l) are per-lane scalars and the rescale of the
// output accumulator is a scalar multiply.  The output is accumulated
// transposed too, O^T = V^T P^T, with V^T fragments from an LDS copy of
// the V tile stored d-major (or, with STAGES 4, of the key-major V tile
// through ds_read_b64_tr_b16); the probabilities never leave registers:
// the MFMA's k index (the key) follows the accumulator layout of S^T, and
// the V^T fragment is read in that same key order.

#define RPW (BM / NW)
#define QB (RPW / MF)
#define NTS (64 * NW)
#define NT (NTS * SPLITS)
#define NBUF (STAGES > 1 ? 2 : 1)      // register-staged paths
// direct-to-LDS paths: ring slots per operand (two per split with several
// splits)
#define RING (STAGES == 5 ? 4 * SPLITS : SPLITS > 1 ? 2 * SPLITS : 3)
#define KB (BN / MF)
#define DB (AD / MF)
#define NQT ((AS + BM - 1) / BM)
#define NKT ((AS + BN - 1) / BN)           // key tiles of the sequence
#define RAGGED_S ((AS % BM) != 0 || (AS % BN) != 0)
#define CPR (AD / 8)
#define RPL ((16 / CPR) > 0 ? (16 / CPR) : 1)
#define SWZ (CPR < 16 ? CPR : 16)
// Lazy rescale: the running max moves (and O, l are rescaled) only when a
// score exceeds it by more than 2^RESCALE_LOG2; stale maxima keep every
// probability below 2^RESCALE_LOG2, exact in fp32 and in bf16.
#define RESCALE_LOG2 8.0f
// V^T tile: d-major rows of BN keys, padded to VTS elements.  Columns hold
// the keys in the order the P^T fragments use (vcol), so one 16-byte read
// gives a lane its 8 keys; the padding (16 for the 16x16 MFMA shape, 8 for
// 32x32) keeps those reads and the 8-byte block stores free of LDS bank
// conflicts.
#define VTS (BN + (MF == 16 ? 16 : 8))
#define K_LOADS ((BN * AD / VEC + NTS - 1) / NTS)
#define V_BLKS ((BN * AD / 32 + NTS - 1) / NTS)
#define KT_ELEMS (BN * AD)
#define VT_ELEMS (AD * VTS)
#define LDS_ELEMS (SPLITS * NBUF * (KT_ELEMS + VT_ELEMS))
// Key-major V tile (STAGES 4): 16-byte chunk c of key row r sits at chunk
// c ^ vswz(r); for 16 consecutive rows the two chunks a transposing read
// takes from each row land on distinct banks.
#define VSWZ(r) ((2 * (r)) & (CPR - 1))
// merge area per partner wave: m and l of its QB * MF queries, then its
// output accumulators lane by lane
#define WSLOT (QB * 2 * MF + QB * DB * ACCN * 64)

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

struct AttnArgs {
    const bf16_t *Q;
    const bf16_t *K;
    const bf16_t *V;
    bf16_t *O;
    float *P;          // partial states of cut query tiles (CHUNK > 0)
};

// XOR swizzle of 16-byte chunks within a K-tile row.  The XOR value depends
// on the row modulo 16 * RPL only, so rows r and r + 16 k share it and a
// fragment offset computed once per lane serves every key block.
__device__ __forceinline__ int kswz(int row, int chunk) {
    return row * AD + ((chunk ^ ((row / RPL) % SWZ)) << 3);
}

__device__ __forceinline__ accT mfma(const bf16x8 &a, const bf16x8 &b, const accT &c) {
#if MF == 16
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
#else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
#endif
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32
__device__ __forceinline__ unsigned pack2(float a, float b) {
    return __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

// Column of key `key` (a multiple of 4: one group of 4 keys) in the V^T tile.
// A lane's P^T fragment for one MFMA k-step holds two groups of 4 keys
// (16 apart for 16x16, 8 apart for 32x32); this interleave makes them
// adjacent.
__device__ __forceinline__ int vcol(int key) {
#if MF == 16
    const int g4 = (key & 31) >> 2;            // 4h + g
    return (key & ~31) + 4 * (2 * (g4 & 3) + (g4 >> 2));
#else
    const int g4 = (key & 15) >> 2;            // 2t + g
    return (key & ~15) + 4 * (2 * (g4 & 1) + (g4 >> 1));
#endif
}

// Key offset (within an MF-key block) of accumulator element r of `lane`.
__device__ __forceinline__ int key_of(int r, int lane) {
#if MF == 16
    return 4 * (lane >> 4) + r;
#else
    return (r >> 2) * 8 + 4 * (lane >> 5) + (r & 3);
#endif
}

// Reductions across the lane groups that hold the other keys of a query:
// lanes l ^ 16 and l ^ 32 (16x16 MFMA) or l ^ 32 (32x32).  v_permlane16_swap
// and v_permlane32_swap (VALU, no LDS round trip) hand every lane the pair
// {v[l], v[l ^ 16]} (resp. l ^ 32) in the same order on both lanes, so the
// reduced value is bit-identical across the lanes of a query.
// The swaps are issued from inline assembly: the compiler's intrinsic for
// them returns the pair, but its optimiser folds the second result into the
// first, which silently drops the partner lane from the reduction.  Both
// registers start as copies of v; the swap and the max (or add) of the pair
// share one asm block, so the compiler adds no NaN-quieting copies around
// the max.  s_nop 1 before each swap and s_nop 0 after it give the wait
// states between a VALU write and the swap's read, and between the swap's
// write and the next VALU read.
#define RC_PAIR_OP(swap, op)                                                              \
    "s_nop 1\n\t" swap " %0, %1\n\ts_nop 0\n\t" op " %0, %0, %1"

__device__ __forceinline__ float group_max(float v) {
    unsigned x = __builtin_bit_cast(unsigned, v), y = x;
#if MF == 16
    asm volatile(RC_PAIR_OP("v_permlane16_swap_b32", "v_max_f32") : "+v"(x), "+v"(y));
    y = x;
#endif
    asm volatile(RC_PAIR_OP("v_permlane32_swap_b32", "v_max_f32") : "+v"(x), "+v"(y));
    return __builtin_bit_cast(float, x);
}

__device__ __forceinline__ float group_sum(float v) {
    unsigned x = __builtin_bit_cast(unsigned, v), y = x;
#if MF == 16
    asm volatile(RC_PAIR_OP("v_permlane16_swap_b32", "v_add_f32") : "+v"(x), "+v"(y));
    y = x;
#endif
    asm volatile(RC_PAIR_OP("v_permlane32_swap_b32", "v_add_f32") : "+v"(x), "+v"(y));
    return __builtin_bit_cast(float, x);
}

// Key tiles seen by query tile t, and the number of work items it is cut into.
constexpr int tiles_of(int t) {
    return CAUSAL ? ((t * BM + BM - 1) / BN + 1 < NKT ? (t * BM + BM - 1) / BN + 1 : NKT) : NKT;
}
constexpr int chunks_of(int t) { return CHUNK > 0 ? (tiles_of(t) + CHUNK - 1) / CHUNK : 1; }
constexpr int items_per_head() {
    int n = 0;
    for (int t = 0; t < NQT; ++t) n += chunks_of(t);
    return n;
}
constexpr int max_chunks() {
    int n = 1;
    for (int t = 0; t < NQT; ++t) n = chunks_of(t) > n ? chunks_of(t) : n;
    return n;
}
// Query tile at position k of the launch order: 0 in order, 1 longest
// first, 2 paired (k and k + NQT / 2 take tiles NQT - 1 - k and k).
constexpr int order_tile(int k) {
    return ORDER == 1 ? NQT - 1 - k : ORDER == 2 ? (k < NQT / 2 ? NQT - 1 - k : k - NQT / 2) : k;
}

// Row of Q (or of K and V) that query (key) row q reads: rows past the
// sequence read its last row, whose results are masked or never stored.
__device__ __forceinline__ int qrow(int q) { return RAGGED_S && q >= AS ? AS - 1 : q; }

// Exponential weight of a state with maximum x relative to the joint maximum
// mt >= x; a state that saw no key (x = mt = -inf) gets weight 1 on its zero
// sums instead of a NaN.
__device__ __forceinline__ float rel_weight(float x, float mt) {
    return x == mt ? 1.0f : __builtin_amdgcn_exp2f(x - mt);
}

// Normalise the transposed output accumulators and store the bf16 rows.
__device__ __forceinline__ void store_out(bf16_t *O, size_t base, int q0w, int lane,
                                          const accT (&o)[QB][DB], const float (&l)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int q = q0w + qb * MF + lane % MF;
        if (RAGGED_S && q >= AS) continue;
        const float inv = 1.0f / l[qb];
        bf16_t *orow = O + base + (size_t)q * AD;
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

extern "C" __global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
void rc_attention(AttnArgs args) {
#if STAGES >= 4
    // ring slots: K tiles in slots 0 .. RING - 1, V tiles after them (one
    // block, reused for the merge of two splits' states at the end)
    __shared__ __attribute__((aligned(16))) bf16_t ring[2 * RING][KT_ELEMS];
    bf16_t *const K0 = ring[0], *const K1 = ring[1], *const K2 = ring[2];
    bf16_t *const V0 = ring[RING], *const V1 = ring[RING + 1], *const V2 = ring[RING + 2];
#if RING >= 4
    bf16_t *const K3 = ring[3], *const V3 = ring[RING + 3];
#endif
    bf16_t *const smem = ring[0];
#else
    // one LDS block: per split, NBUF K tiles then NBUF V^T tiles; reused for
    // the merge of the splits' states at the end
    __shared__ __attribute__((aligned(16))) bf16_t smem[LDS_ELEMS];
#endif

    // wave index made wave-uniform: the row group and split it selects feed
    // scalar operands (direct-to-LDS addresses) and scalar branches
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int rg = wave % NW, sp = wave / NW, tids = tid % NTS;
    bf16_t *const Kbase = smem + sp * NBUF * (KT_ELEMS + VT_ELEMS);
    bf16_t *const Vbase = Kbase + NBUF * KT_ELEMS;
    // work item: head bh, j-th item of its launch order (ORDER 0 keeps a
    // head's items together, 1 and 2 interleave the heads)
    const int bid = blockIdx.x;
#if ORDER == 0
    const int bh = bid / items_per_head();
    int j = bid % items_per_head();
#else
    const int bh = bid % (AB * AH);
    int j = bid / (AB * AH);
#endif
    int qt = order_tile(j), ch = 0;
#if CHUNK > 0
    for (int k = 0; k < NQT; ++k) {
        const int t = order_tile(k), n = chunks_of(t);
        if (j < n) {
            qt = t;
            ch = j;
            break;
        }
        j -= n;
    }
#endif
    const int q0 = qt * BM;
    const int q0w = q0 + rg * RPW;
    const size_t base = (size_t)bh * AS * AD;
    // key tiles kt0 .. kt0 + n_kt - 1; the loops below count kt from 0
    const int kt0 = ch * CHUNK;
    const int n_kt = CHUNK > 0 ? min(CHUNK, tiles_of(qt) - kt0) : tiles_of(qt);
#if STAGES >= 4
    // Direct-to-LDS loads: one global_load_lds_dwordx4 moves 64 lanes x 16 B
    // into 1 KiB of LDS at a wave-uniform base (M0), lane i at byte 16 i.
    // The swizzles are applied by choosing which global chunk each lane
    // fetches: LDS chunk c of a tile holds row c / CPR, logical chunk
    // (c % CPR) XOR the row's swizzle (an involution).
    //
    // The loads are issued from inline assembly, so the compiler's
    // wait-count bookkeeping does not see them: it cannot tell, across the
    // loop's back edge, which ring buffer a load fills, and would otherwise
    // drain every load before each LDS read.  The kernel's own waits below
    // order the ring.  The compiler's waits for its own loads stay correct:
    // extra loads in flight only make a vmcnt(n) wait longer.
    // Each split's NW waves load that split's tiles.
    constexpr int WL = BN * AD / 512 / NW;            // wave-loads per wave and operand
    unsigned k_src[WL], v_src[WL];                    // byte offsets within a tile
    int kv_row[RAGGED_S ? WL : 1];                    // key row of each offset
#pragma unroll
    for (int j = 0; j < WL; ++j) {
        const int c = (rg * WL + j) * 64 + lane;
        const int row = c / CPR, pc = c % CPR;
        k_src[j] = 2u * (row * AD + ((pc ^ ((row / RPL) % SWZ)) << 3));
        v_src[j] = 2u * (row * AD + ((pc ^ VSWZ(row)) << 3));
        if (RAGGED_S) kv_row[RAGGED_S ? j : 0] = row;
    }
    // LDS byte addresses of the ring buffers and this wave's first 1 KiB
    typedef __attribute__((address_space(3))) bf16_t *lds_p;
    const unsigned wl0 = (unsigned)__builtin_amdgcn_readfirstlane(rg) * WL * 1024u;
    const unsigned ka0 = (unsigned)(size_t)(lds_p)ring[0] + wl0;
    // K and V slot b (the slots are consecutive KT_ELEMS blocks)
    auto KA = [&](int b) { return ka0 + (unsigned)b * (KT_ELEMS * 2u); };
    auto VA = [&](int b) { return ka0 + (unsigned)(RING + b) * (KT_ELEMS * 2u); };
    auto dma = [&](const bf16_t *gbase, unsigned off, unsigned lds_addr) {
        asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                     :: "v"(off), "s"(gbase), "s"(lds_addr) : "memory", "m0");
    };
    // tile kt into ring buffer b
    auto gload_lds = [&](int kt, int b) {
        const bf16_t *Kg = args.K + base + (size_t)(kt0 + kt) * BN * AD;
        const bf16_t *Vg = args.V + base + (size_t)(kt0 + kt) * BN * AD;
        const int kvalid = AS - (kt0 + kt) * BN;     // wave-uniform
        if (RAGGED_S && kvalid < BN) {
            // last, partial tile: rows past the sequence fetch its last row
#pragma unroll
            for (int j = 0; j < WL; ++j) {
                const unsigned back = 2u * AD * (unsigned)max(kv_row[RAGGED_S ? j : 0] - (kvalid - 1), 0);
                dma(Kg, k_src[j] - back, KA(b) + j * 1024u);
            }
#pragma unroll
            for (int j = 0; j < WL; ++j) {
                const unsigned back = 2u * AD * (unsigned)max(kv_row[RAGGED_S ? j : 0] - (kvalid - 1), 0);
                dma(Vg, v_src[j] - back, VA(b) + j * 1024u);
            }
            return;
        }
#pragma unroll
        for (int j = 0; j < WL; ++j) dma(Kg, k_src[j], KA(b) + j * 1024u);
#pragma unroll
        for (int j = 0; j < WL; ++j) dma(Vg, v_src[j], VA(b) + j * 1024u);
    };
#if STAGES == 5
    // split sp's first three tiles (sp, sp + SPLITS, sp + 2 SPLITS) are in
    // flight while Q is read, in the split's slots 4 sp .. 4 sp + 2
#pragma unroll
    for (int u = 0; u < 3; ++u)
        if (SPLITS * u + sp < n_kt) gload_lds(SPLITS * u + sp, 4 * sp + u);
#elif SPLITS == 1
    // the first RING - 1 key tiles are in flight while Q is read
#pragma unroll
    for (int t = 0; t < RING - 1; ++t)
        if (t < n_kt) gload_lds(t, t);
#else
    // split sp's first tile (tile sp) is in flight while Q is read
    if (sp < n_kt) gload_lds(sp, sp);
#endif
#endif
    bf16x8 qf[QB][AD / KSTEP];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int ks = 0; ks < AD / KSTEP; ++ks)
            qf[qb][ks] = *(const bf16x8 *)(args.Q + base + (size_t)qrow(q0w + qb * MF + lane % MF) * AD +
                                           ks * KSTEP + 8 * (lane / MF));
#if STAGES >= 4
    // Consume Q here so that the compiler's wait for it (a full vmcnt drain,
    // which also lands tiles 0 and 1) sits before the loop rather than in it.
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int ks = 0; ks < AD / KSTEP; ++ks) asm volatile("" :: "v"(qf[qb][ks]));
    __builtin_amdgcn_s_waitcnt(0x0F70);      // vmcnt(0)
    __syncthreads();
#endif

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


    vecT rk[K_LOADS];
    u32x4 rv[V_BLKS][4];
    // per-lane offset of the K fragment of k-step ks in key block 0
    int koff[AD / KSTEP];
#pragma unroll
    for (int ks = 0; ks < AD / KSTEP; ++ks) koff[ks] = kswz(lane % MF, ks * (KSTEP / 8) + lane / MF);

    auto gload = [&](int kt) {
        const bf16_t *Kg = args.K + base + (size_t)(kt0 + kt) * BN * AD;
        const bf16_t *Vg = args.V + base + (size_t)(kt0 + kt) * BN * AD;
        // keys of this tile that lie inside the sequence (rows past it load zeros)
        const int kvalid = AS - (kt0 + kt) * BN;
#pragma unroll
        for (int i = 0; i < K_LOADS; ++i) {
            int idx = tids + i * NTS;
            if ((BN * AD / VEC) % NTS == 0 || idx < BN * AD / VEC)
                rk[i] = (!RAGGED_S || idx / (AD / VEC) < kvalid) ? *(const vecT *)(Kg + (size_t)idx * VEC) : vecT{};
        }
#pragma unroll
        for (int i = 0; i < V_BLKS; ++i) {
            int blk = tids + i * NTS;
            if ((BN * AD / 32) % NTS == 0 || blk < BN * AD / 32) {
                int kr = (blk % (BN / 4)) * 4, dc = (blk / (BN / 4)) * 8;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    rv[i][j] = (!RAGGED_S || kr + j < kvalid) ? *(const u32x4 *)(Vg + (size_t)(kr + j) * AD + dc)
                                                             : u32x4{0u, 0u, 0u, 0u};
            }
        }
    };

    auto swrite = [&](int s) {
        bf16_t *const Ks = Kbase + s * KT_ELEMS;
        bf16_t *const Vt = Vbase + s * VT_ELEMS;
#pragma unroll
        for (int i = 0; i < K_LOADS; ++i) {
            int idx = tids + i * NTS;
            if ((BN * AD / VEC) % NTS == 0 || idx < BN * AD / VEC) {
                int row = idx / (AD / VEC), c = (idx % (AD / VEC)) * VEC;
                *(vecT *)(Ks + kswz(row, c >> 3) + (c & 7)) = rk[i];
            }
        }
#pragma unroll
        for (int i = 0; i < V_BLKS; ++i) {
            int blk = tids + i * NTS;
            if ((BN * AD / 32) % NTS == 0 || blk < BN * AD / 32) {
                int kr = (blk % (BN / 4)) * 4, dc = (blk / (BN / 4)) * 8;
                const int col = vcol(kr);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    // column d = dc + j of keys kr .. kr+3: one byte permute per
                    // pair of keys picks the low (j even) or high (j odd) halves
                    const unsigned sel = (j & 1) ? 0x07060302u : 0x05040100u;
                    const int c = j >> 1;
                    u32x2 w;
                    w[0] = __builtin_amdgcn_perm(rv[i][1][c], rv[i][0][c], sel);
                    w[1] = __builtin_amdgcn_perm(rv[i][3][c], rv[i][2][c], sel);
                    *(u32x2 *)(Vt + (dc + j) * VTS + col) = w;
                }
            }
        }
    };

    // true when every key of tile kt is masked for this wave's queries
    auto skipped = [&](int kt) {
#if CAUSAL
        return (kt0 + kt) * BN > q0w + RPW - 1;
#else
        (void)kt;
        return false;
#endif
    };

    // S^T = K Q^T of tile kt (LDS buffer s) for every query block; each K
    // fragment is read once
    auto scores_at = [&](const bf16_t *Ks, accT (&sc)[QB][KB]) {
#if STAGES >= 4
        // even and odd k-steps accumulate separately and are added at the
        // end: dependent MFMA chains half as long
        accT sc2[QB][KB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) sc[qb][kb][r] = sc2[qb][kb][r] = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int ks = 0; ks < AD / KSTEP; ++ks) {
                bf16x8 kf = *(const bf16x8 *)(Ks + kb * MF * AD + koff[ks]);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) {
                    if (ks & 1) sc2[qb][kb] = mfma(kf, qf[qb][ks], sc2[qb][kb]);
                    else sc[qb][kb] = mfma(kf, qf[qb][ks], sc[qb][kb]);
                }
            }
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) sc[qb][kb] += sc2[qb][kb];
#else
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
                bf16x8 kf = *(const bf16x8 *)(Ks + kb * MF * AD + koff[ks]);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) sc[qb][kb] = mfma(kf, qf[qb][ks], sc[qb][kb]);
            }
#endif
    };
    auto scores = [&](int s, accT (&sc)[QB][KB]) { scores_at(Kbase + s * KT_ELEMS, sc); };

#if STAGES >= 4
    // per-lane offsets (elements, relative to the V buffer) of the row and
    // column this lane addresses in the transposing read of key block j,
    // half h, d block db: row 32 j + 16 h + 4 (lane / 16) + (lane % 16) / 4,
    // columns 16 db + 4 (lane % 4) .. + 3 (16x16 MFMA only)
    int voff[DB];
    {
        const int vr = 4 * (lane >> 4) + ((lane & 15) >> 2);
#pragma unroll
        for (int db = 0; db < DB; ++db)
            voff[db] = vr * AD + (((2 * db + ((lane & 3) >> 1)) ^ VSWZ(vr)) << 3) + (lane & 1) * 4;
    }
#endif

    // online softmax of tile kt's scores and O^T += V^T P^T (V^T from buffer s)
    auto softmax_pv_at = [&](int kt, const bf16_t *Vt, accT (&sc)[QB][KB]) {
#if STAGES >= 4
        // the tile's V^T fragments (at most 16 x 16 B per lane) are read
        // ahead of their MFMAs: the first NPRE d-blocks before the softmax,
        // which does not need them, so their LDS latency overlaps the
        // exponentials and reductions, the rest together before the first
        // P.V MFMA.  With two key splits the workgroup's waves must fit four
        // per SIMD (128 registers), which leaves room for half of them
        // across the softmax.
        typedef short v4i16 __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) v4i16 *lds_v4p;
        constexpr bool VPRE = (BN / KSTEP) * DB <= 16;
        constexpr int NPRE = SPLITS == 1 ? DB : DB / 2;
        bf16x8 vpre[VPRE ? BN / KSTEP : 1][VPRE ? DB : 1];
        auto read_vt = [&](int j, int db) {
            const bf16_t *const vp = Vt + voff[db] + 32 * j * AD;
            const v4i16 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4p)(vp));
            const v4i16 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4p)(vp + 16 * AD));
            return __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
        };
        if (VPRE) {
#pragma unroll
            for (int j = 0; j < (VPRE ? BN / KSTEP : 1); ++j)
#pragma unroll
                for (int db = 0; db < (VPRE ? NPRE : 1); ++db) vpre[j][db] = read_vt(j, db);
        }
#endif
        // online softmax, one query per lane; m is kept in log2 units and the
        // scale is folded into the exponent's fused multiply-add
#if CAUSAL
        // only a tile that crosses this wave's diagonal needs the mask
        const bool diag = (kt0 + kt) * BN + BN - 1 > q0w;
#else
        // only the last tile of a ragged sequence holds keys past its end
        const bool tail = RAGGED_S && (kt0 + kt) * BN + BN > AS;
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
                        if ((kt0 + kt) * BN + kb * MF + key_of(r, lane) > q) sc[qb][kb][r] = -__builtin_inff();
            }
#else
            if (tail) {
#pragma unroll
                for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                    for (int r = 0; r < ACCN; ++r)
                        if ((kt0 + kt) * BN + kb * MF + key_of(r, lane) >= AS) sc[qb][kb][r] = -__builtin_inff();
            }
#endif
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) mx = fmaxf(mx, sc[qb][kb][r]);
            mx = group_max(mx) * SCALE_LOG2;
            if (__builtin_amdgcn_ballot_w64(mx > m[qb] + RESCALE_LOG2) != 0) {
                const float mnew = fmaxf(m[qb], mx);
                const float alpha = __builtin_amdgcn_exp2f(m[qb] - mnew);
                l[qb] *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int r = 0; r < ACCN; ++r) o[qb][db][r] *= alpha;
                m[qb] = mnew;
            }
            const float mnew = m[qb];
            float ps = 0.f;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) {
                    float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][kb][r], SCALE_LOG2, -mnew));
                    sc[qb][kb][r] = p;
                    ps += p;
                }
            // per-lane partial row sums; the lanes of a query apply the same
            // rescale factors, so they are added across lanes once, at the end
            l[qb] += ps;
        }
        // O^T += V^T P^T, KSTEP keys per MFMA; each V^T fragment is read once
#pragma unroll
        for (int j = 0; j < BN / KSTEP; ++j) {
            bf16x8 pf[QB];
#if MF == 16
            const int c0 = 32 * j + 8 * (lane >> 4);
#else
            const int kb = j >> 1, hf = (j & 1) * 8;
            const int c0 = 16 * j + 8 * (lane >> 5);
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
#if STAGES >= 4
            if (VPRE) {
#pragma unroll
                for (int db = NPRE; db < (VPRE ? DB : 0); ++db) vpre[VPRE ? j : 0][db] = read_vt(j, db);
            }
#endif
#pragma unroll
            for (int db = 0; db < DB; ++db) {
#if STAGES >= 4
                const bf16x8 vf = VPRE ? vpre[VPRE ? j : 0][VPRE ? db : 0] : read_vt(j, db);
                (void)c0;
#else
                const int drow = db * MF + lane % MF;
                const bf16x8 vf = *(const bf16x8 *)(Vt + drow * VTS + c0);
#endif
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) o[qb][db] = mfma(vf, pf[qb], o[qb][db]);
            }
        }
    };

    auto softmax_pv = [&](int kt, int s, accT (&sc)[QB][KB]) { softmax_pv_at(kt, Vbase + s * VT_ELEMS, sc); };

    auto compute = [&](int kt, int s) {
        if (skipped(kt)) return;
        accT sc[QB][KB];
        scores(s, sc);
        softmax_pv(kt, s, sc);
    };

    // split sp visits key tiles sp, sp + SPLITS, ...; every wave runs the same
    // number of iterations so the workgroup barriers line up
    const int n_it = (n_kt + SPLITS - 1) / SPLITS;
#if STAGES == 4 && SPLITS > 1
    (void)compute;
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    // The splits share a ring of 2 x SPLITS slots: iteration i computes tile
    // SPLITS i + split from slot SPLITS (i % 2) + split, while each split
    // loads its next tile into the same slot of the other half of the ring.
    // That half was last read in iteration i - 1, before the last barrier.
    auto body = [&](int it, int pair) {
        const int kt = SPLITS * it + sp, nk = kt + SPLITS;
        if (nk < n_kt) gload_lds(nk, SPLITS - pair + sp);
        if (kt < n_kt && !skipped(kt)) {
            accT sc[QB][KB];
            scores_at(ring[pair + sp], sc);
            softmax_pv_at(kt, ring[RING + pair + sp], sc);
        }
        WAIT_VM(0);                // this wave's share of the next tiles has landed
        __builtin_amdgcn_s_waitcnt(0xC07F);      // lgkmcnt(0): this wave's LDS reads are done
        asm volatile("s_barrier" ::: "memory");
    };
    for (int it = 0; it < n_it; it += 2) {
        body(it, 0);
        if (it + 1 < n_it) body(it + 1, SPLITS);
    }
#undef WAIT_VM
#elif STAGES == 4
    (void)n_it;
    (void)compute;
    // s_waitcnt with only the vector-memory count constrained (expcnt and
    // lgkmcnt at their maxima): at most n loads of this wave still in flight
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    // tile kt sits in buffer kt % 3; buffer (kt + 2) % 3 held tile kt - 1,
    // finished before the last barrier, and receives tile kt + 2
    auto body = [&](int kt, const bf16_t *kc, const bf16_t *vc, int fill) {
        if (kt + 2 < n_kt) gload_lds(kt + 2, fill);
        if (!skipped(kt)) {
            accT sc[QB][KB];
            scores_at(kc, sc);
            softmax_pv_at(kt, vc, sc);
        }
        if (kt + 2 < n_kt) {
            WAIT_VM(2 * WL);       // tile kt + 1 has landed; tile kt + 2 may be in flight
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
    for (int kt = 0; kt < n_kt; kt += 3) {
        body(kt, K0, V0, 2);
        if (kt + 1 < n_kt) body(kt + 1, K1, V1, 0);
        if (kt + 2 < n_kt) body(kt + 2, K2, V2, 1);
    }
#undef WAIT_VM
#elif STAGES == 5
    (void)compute;
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    // Software pipeline over a ring of four K/V tiles per key split.
    // Iteration kt (of a split's tiles) runs two
    // phases, each pairing matrix work with vector work that does not depend
    // on it, so the MFMAs execute while the VALU exponentiates:
    //   phase 1: S^T of tile kt + 1 (MFMA)  |  exponentials, row sums and
    //            bf16 packing of tile kt's probabilities (VALU)
    //   phase 2: O^T += V^T P^T of tile kt (MFMA)  |  row maximum of tile
    //            kt + 1's scores (VALU)
    // The order inside each phase is fixed with scheduling-group barriers.
    // The lazy rescale of tile kt (rare) sits between iterations, the causal
    // mask (only a wave's last tile crosses its diagonal) between the phases.
    // Row sums are kept per lane and reduced across lane groups once, after
    // the loop: every lane of a query applies the same rescale factors.
    //
    // Split sp takes the key tiles sp, sp + SPLITS, ...; its j-th tile
    // (tile SPLITS j + sp) sits in ring slot 4 sp + j % 4.  Iteration j reads
    // K of the split's tile j + 1 and V of its tile j and fills slot
    // 4 sp + (j + 3) % 4, which held its tile j - 1 (whose K was read in
    // iteration j - 2, its V in j - 1, both before the last barrier).  Every
    // wave runs n_it iterations, so the barriers line up across splits.
    auto gt = [&](int j) { return SPLITS * j + sp; };        // tile of the split's j-th
    auto local_count = [&](int n) { return n > sp ? (n - sp - 1) / SPLITS + 1 : 0; };
    const int n_loc = local_count(n_kt);
#if CAUSAL
    // the split's tiles below the last key tile that holds a key visible to
    // this wave's rows
    const int nact = local_count(max(0, min(n_kt, (q0w + RPW - 1) / BN - kt0 + 1)));
#else
    const int nact = n_loc;
#endif
    bf16_t *const Ks = ring[4 * sp], *const Vs = ring[RING + 4 * sp];   // the split's slot 0
    constexpr int NKS = AD / KSTEP;            // k-steps of the score product
    constexpr int NPJ = BN / KSTEP;            // k-steps of the P V product
    constexpr int MF1 = KB * NKS * QB;         // phase-1 MFMAs
    constexpr int MF2 = NPJ * DB * QB;         // phase-2 MFMAs
    constexpr int VALU1 = QB * KB * ACCN * 3 + NPJ * QB * 4;   // phase-1 VALU (approx.)
    constexpr int V1_PER = (VALU1 + MF1 - 1) / MF1;
    constexpr int DS1 = KB * NKS + 2 * NPJ * DB;            // phase-1 LDS reads
    constexpr int DS1_PER = (DS1 - KB * NKS + MF1 - 1) / MF1;
    typedef short v4i16 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) v4i16 *lds_v4p;
    auto needs_mask = [&](int kt) {
#if CAUSAL
        return (kt0 + kt) * BN + BN - 1 > q0w;
#else
        return RAGGED_S && (kt0 + kt) * BN + BN > AS;
#endif
    };
    auto mask = [&](int kt, accT (&sc)[QB][KB]) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
#if CAUSAL
            const int q = q0w + qb * MF + lane % MF;
#else
            const int q = AS - 1;      // keys past the sequence
#endif
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r)
                    if ((kt0 + kt) * BN + kb * MF + key_of(r, lane) > q) sc[qb][kb][r] = -__builtin_inff();
        }
    };
    // row maximum of a tile in log2 units, identical on every lane of a query
    auto tile_max = [&](const accT (&sc)[QB][KB], float (&mx)[QB]) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float v = -__builtin_inff();
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) v = fmaxf(v, sc[qb][kb][r]);
            mx[qb] = group_max(v) * SCALE_LOG2;
        }
    };
    auto rescale = [&](const float (&mx)[QB]) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
            if (__builtin_amdgcn_ballot_w64(mx[qb] > m[qb] + RESCALE_LOG2) != 0) {
                const float mnew = fmaxf(m[qb], mx[qb]);
                const float alpha = __builtin_amdgcn_exp2f(m[qb] - mnew);
                l[qb] *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int r = 0; r < ACCN; ++r) o[qb][db][r] *= alpha;
                m[qb] = mnew;
            }
    };
    // probabilities of a tile, packed into the P^T fragments of the P V product
    auto probs = [&](accT (&sc)[QB][KB], bf16x8 (&pf)[NPJ][QB]) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float ps = l[qb];
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) {
                    const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][kb][r], SCALE_LOG2, -m[qb]));
                    sc[qb][kb][r] = p;
                    ps += p;
                }
            l[qb] = ps;
        }
#pragma unroll
        for (int j = 0; j < NPJ; ++j)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                u32x4 pw;
                pw[0] = pack2(sc[qb][2 * j][0], sc[qb][2 * j][1]);
                pw[1] = pack2(sc[qb][2 * j][2], sc[qb][2 * j][3]);
                pw[2] = pack2(sc[qb][2 * j + 1][0], sc[qb][2 * j + 1][1]);
                pw[3] = pack2(sc[qb][2 * j + 1][2], sc[qb][2 * j + 1][3]);
                pf[j][qb] = __builtin_bit_cast(bf16x8, pw);
            }
    };
    auto read_k = [&](const bf16_t *Ks, bf16x8 (&kf)[KB][NKS]) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) kf[kb][ks] = *(const bf16x8 *)(Ks + kb * MF * AD + koff[ks]);
    };
    auto read_v = [&](const bf16_t *Vt, bf16x8 (&vf)[NPJ][DB]) {
#pragma unroll
        for (int j = 0; j < NPJ; ++j)
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const bf16_t *const vp = Vt + voff[db] + 32 * j * AD;
                const v4i16 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4p)(vp));
                const v4i16 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4p)(vp + 16 * AD));
                vf[j][db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
            }
    };
    auto score_mfmas = [&](const bf16x8 (&kf)[KB][NKS], accT (&sc)[QB][KB]) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) sc[qb][kb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) sc[qb][kb] = mfma(kf[kb][ks], qf[qb][ks], sc[qb][kb]);
    };
    auto pv_mfmas = [&](const bf16x8 (&vf)[NPJ][DB], const bf16x8 (&pf)[NPJ][QB]) {
#pragma unroll
        for (int j = 0; j < NPJ; ++j)
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int qb = 0; qb < QB; ++qb) o[qb][db] = mfma(vf[j][db], pf[j][qb], o[qb][db]);
    };

    accT sc_a[QB][KB], sc_b[QB][KB];
    float mx[QB];
    if (nact > 0) {
        bf16x8 kf[KB][NKS];
        read_k(Ks, kf);
        score_mfmas(kf, sc_a);
        if (needs_mask(gt(0))) mask(gt(0), sc_a);
        tile_max(sc_a, mx);
    }
    // Phase 1 as straight-line code (the scheduling groups act within one
    // basic block); MASKED applies the causal mask to the successor tile's
    // scores (tile ktn).
    auto phase1 = [&](auto masked, int ktn, accT (&cur)[QB][KB], accT (&nxt)[QB][KB], const bf16_t *kn,
                      const bf16_t *vc, bf16x8 (&vf)[NPJ][DB], bf16x8 (&pf)[NPJ][QB]) {
        bf16x8 kf[KB][NKS];
        // distinct markers keep the compiler from hoisting the variants'
        // common code above the branch that selects the variant
        if (decltype(masked)::value) asm volatile("; pipelined tile, masked successor");
        else asm volatile("; pipelined tile");
        read_k(kn, kf);
        read_v(vc, vf);
        probs(cur, pf);
        score_mfmas(kf, nxt);
        __builtin_amdgcn_sched_group_barrier(0x100, KB * NKS, 0);    // K fragment reads
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
#pragma unroll
        for (int i = 0; i < MF1; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, V1_PER, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, DS1_PER, 0);
        }
        if (decltype(masked)::value) {
            mask(ktn, nxt);
            // keep the mask inside this variant (not merged into the common
            // block as selects that every tile would execute)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
                for (int kb = 0; kb < KB; ++kb) asm volatile("" : "+v"(nxt[qb][kb]));
        }
    };
    auto body = [&](int j, accT (&cur)[QB][KB], accT (&nxt)[QB][KB], const bf16_t *kn,
                    const bf16_t *vc, int fill) {
        if (j + 3 < n_loc) gload_lds(gt(j + 3), 4 * sp + fill);
        if (j < nact) {
            rescale(mx);
            bf16x8 vf[NPJ][DB], pf[NPJ][QB];
            if (j + 1 < nact) {
                if (needs_mask(gt(j + 1))) phase1(IntC<1>{}, gt(j + 1), cur, nxt, kn, vc, vf, pf);
                else phase1(IntC<0>{}, gt(j + 1), cur, nxt, kn, vc, vf, pf);
            } else {
                // the wave's last tile: no successor to overlap with
                asm volatile("; last tile");
                read_v(vc, vf);
                probs(cur, pf);
            }
            // phase 2 (one block for every variant, so each output
            // accumulator has a single MFMA site); after the last tile the
            // maximum is of stale scores and unused
            pv_mfmas(vf, pf);
            tile_max(nxt, mx);
#pragma unroll
            for (int i = 0; i < MF2; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
                __builtin_amdgcn_sched_group_barrier(0x002, 2, 1);
            }
        }
        if (j + 3 < n_loc) {
            WAIT_VM(2 * WL);       // tiles up to j + 2 have landed; j + 3 may be in flight
        } else {
            WAIT_VM(0);
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);      // lgkmcnt(0): this wave's LDS reads are done
        asm volatile("s_barrier" ::: "memory");
    };
    // slot u of the split: K at Ks + u KT_ELEMS, V at Vs + u KT_ELEMS
    for (int j = 0; j < n_it; j += 4) {
        body(j, sc_a, sc_b, Ks + KT_ELEMS, Vs, 3);
        if (j + 1 < n_it) body(j + 1, sc_b, sc_a, Ks + 2 * KT_ELEMS, Vs + KT_ELEMS, 0);
        if (j + 2 < n_it) body(j + 2, sc_a, sc_b, Ks + 3 * KT_ELEMS, Vs + 2 * KT_ELEMS, 1);
        if (j + 3 < n_it) body(j + 3, sc_b, sc_a, Ks, Vs + 3 * KT_ELEMS, 2);
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l[qb] = group_sum(l[qb]);
#undef WAIT_VM
#elif STAGES == 3
    // Software pipeline: iteration i issues the score MFMAs of tile i + 1
    // (K from the other buffer) ahead of the softmax of tile i, so the matrix
    // unit works while the vector unit exponentiates; then P V of tile i.
    // Buffer i & 1 is refilled with tile i + 2 between two barriers.
    accT sc_a[QB][KB], sc_b[QB][KB];
    if (sp < n_kt) {
        gload(sp);
        swrite(0);
    }
    if (sp + SPLITS < n_kt) {
        gload(sp + SPLITS);
        swrite(1);
    }
    __syncthreads();
    if (sp < n_kt && !skipped(sp)) scores(0, sc_a);
    auto step = [&](int it, accT (&cur)[QB][KB], accT (&nxt)[QB][KB]) {
        const int kt = it * SPLITS + sp, kn = kt + SPLITS, k2 = kn + SPLITS;
        if (k2 < n_kt) gload(k2);
        if (kn < n_kt && !skipped(kn)) scores((it + 1) & 1, nxt);
        if (kt < n_kt && !skipped(kt)) softmax_pv(kt, it & 1, cur);
        __syncthreads();
        if (k2 < n_kt) swrite(it & 1);
        __syncthreads();
    };
    for (int it = 0; it < n_it; it += 2) {
        step(it, sc_a, sc_b);
        if (it + 1 < n_it) step(it + 1, sc_b, sc_a);
    }
#elif STAGES == 1
#pragma unroll UNROLL
    for (int it = 0; it < n_it; ++it) {
        const int kt = it * SPLITS + sp;
        if (kt < n_kt) {
            gload(kt);
            swrite(0);
        }
        __syncthreads();
        if (kt < n_kt) compute(kt, 0);
        __syncthreads();
    }
#else
    if (sp < n_kt) {
        gload(sp);
        swrite(0);
    }
    __syncthreads();
#pragma unroll UNROLL
    for (int it = 0; it < n_it; ++it) {
        const int kt = it * SPLITS + sp, nk = kt + SPLITS;
        if (nk < n_kt) gload(nk);
        if (kt < n_kt) compute(kt, it & 1);
        if (nk < n_kt) swrite((it + 1) & 1);
        __syncthreads();
    }
#endif

#if STAGES != 5
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l[qb] = group_sum(l[qb]);
#endif

#if SPLITS > 1
    // merge: splits 1.. publish (m, l, O) in LDS, split 0 folds them in
    float *const cmb = (float *)smem;
    if (sp > 0) {
        float *w = cmb + ((sp - 1) * NW + rg) * WSLOT;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
            if (lane < MF) {
                w[qb * 2 * MF + lane] = m[qb];
                w[qb * 2 * MF + MF + lane] = l[qb];
            }
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) w[QB * 2 * MF + ((qb * DB + db) * ACCN + r) * 64 + lane] = o[qb][db][r];
    }
    __syncthreads();
    if (sp > 0) return;
#pragma unroll
    for (int p = 1; p < SPLITS; ++p) {
        const float *w = cmb + ((p - 1) * NW + rg) * WSLOT;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float mp = w[qb * 2 * MF + lane % MF], lp = w[qb * 2 * MF + MF + lane % MF];
            const float mt = fmaxf(m[qb], mp);
            const float a0 = rel_weight(m[qb], mt), a1 = rel_weight(mp, mt);
            l[qb] = l[qb] * a0 + lp * a1;
            m[qb] = mt;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < ACCN; ++r)
                    o[qb][db][r] = o[qb][db][r] * a0 + w[QB * 2 * MF + ((qb * DB + db) * ACCN + r) * 64 + lane] * a1;
        }
    }
#endif

#if CHUNK > 0
    if (chunks_of(qt) > 1) {
        // one of several items of this query tile: leave the state for the
        // combine kernel, same layout as the split merge area
        float *w = args.P + ((size_t)(bh * NQT + qt) * max_chunks() + ch) * (NW * WSLOT) + rg * WSLOT;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
            if (lane < MF) {
                w[qb * 2 * MF + lane] = m[qb];
                w[qb * 2 * MF + MF + lane] = l[qb];
            }
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < ACCN; ++r) w[QB * 2 * MF + ((qb * DB + db) * ACCN + r) * 64 + lane] = o[qb][db][r];
        return;
    }
#endif
    store_out(args.O, base, q0w, lane, o, l);
}

#if CHUNK > 0
// Merge the partial states of the query tiles that were cut into several
// work items (rescale each to the joint maximum, add, normalise).  One
// workgroup per query tile, one wave per row group, lanes laid out as in
// rc_attention.
extern "C" __global__ __launch_bounds__(64 * NW) void rc_attention_combine(AttnArgs args) {
    const int lane = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const int bh = blockIdx.x / NQT, qt = blockIdx.x % NQT;
    const int nc = chunks_of(qt);
    if (nc == 1) return;
    const float *w = args.P + (size_t)(bh * NQT + qt) * max_chunks() * (NW * WSLOT) + rg * WSLOT;
    accT o[QB][DB];
    float m[QB], l[QB];
    // chunk 0 holds key tile 0, which every query sees: its maximum is finite
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m[qb] = w[qb * 2 * MF + lane % MF];
        l[qb] = w[qb * 2 * MF + MF + lane % MF];
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < ACCN; ++r) o[qb][db][r] = w[QB * 2 * MF + ((qb * DB + db) * ACCN + r) * 64 + lane];
    }
    for (int c = 1; c < nc; ++c) {
        const float *v = w + (size_t)c * (NW * WSLOT);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float mp = v[qb * 2 * MF + lane % MF], lp = v[qb * 2 * MF + MF + lane % MF];
            const float mt = fmaxf(m[qb], mp);
            const float a0 = rel_weight(m[qb], mt), a1 = rel_weight(mp, mt);
            l[qb] = l[qb] * a0 + lp * a1;
            m[qb] = mt;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < ACCN; ++r)
                    o[qb][db][r] = o[qb][db][r] * a0 + v[QB * 2 * MF + ((qb * DB + db) * ACCN + r) * 64 + lane] * a1;
        }
    }
    store_out(args.O, (size_t)bh * AS * AD, qt * BM + rg * RPW, lane, o, l);
}
#endif
