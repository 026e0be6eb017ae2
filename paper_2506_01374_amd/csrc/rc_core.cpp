// Operator descriptors, knob tables, legality, transformations and the
// FLOP / byte model.  Host-only code; no GPU access.
//
// The search space follows the paper's formulation (Sec. 2, Eq. 1): a
// program variant is reached from P0 by a sequence of transformations, each
// of which preserves semantics.  Here a variant is a vector of knob values
// and a transformation sets one knob.  The knob classes are the
// transformation names of App. A (TileSize, Parallel, ComputeLocation,
// Unroll) plus the vectorisation and layout changes named in Sec. 1.
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <string>

#include "rc_internal.h"

namespace rc {

static thread_local std::string g_err;

rc_status fail(rc_status s, const std::string &msg) {
    g_err = msg;
    return s;
}
void clear_error() { g_err.clear(); }

static std::vector<KnobDef> gemm_f32_knobs() {
    return {
        {"tile_m", "TileSize", {16, 32, 64}, 16},
        {"tile_n", "TileSize", {16, 32, 64}, 16},
        {"tile_k", "TileSize", {4, 8, 16, 32}, 4},
        {"waves_m", "Parallel", {1, 2}, 1},
        {"waves_n", "Parallel", {1, 2}, 1},
        {"vec", "Vectorize", {1, 4}, 1},
        {"stages", "ComputeLocation", {1, 2, 3}, 1},
        {"unroll", "Unroll", {1, 2, 4}, 1},
        {"layout", "Layout", {0, 1}, 0},
        {"splits", "Parallel", {1, 2, 4, 8, 16, 32, 64}, 1},   // K splits across workgroups
    };
}

// One bf16 GEMM stage's knobs, names prefixed ("" / "up." / "down.").
static void add_gemm_block(std::vector<KnobDef> &v, const char *const names[12],
                           std::vector<int32_t> tile_n_vals, std::vector<int32_t> tile_k_vals) {
    // 96 and 192 rows fit ragged row groups (MoE experts) of ~3 x 64 rows
    v.push_back({names[0], "TileSize", {16, 32, 64, 96, 128, 192, 256}, 16});
    v.push_back({names[1], "TileSize", tile_n_vals, 16});
    v.push_back({names[2], "TileSize", tile_k_vals, 32});
    v.push_back({names[3], "Parallel", {1, 2, 4}, 1});
    v.push_back({names[4], "Parallel", {1, 2, 4}, 1});
    v.push_back({names[5], "TileSize", {16, 32}, 16});          // MFMA instruction shape
    v.push_back({names[6], "ComputeLocation", {1, 2, 3, 4, 5, 6, 7}, 1});   // LDS staging of the next K tile
    v.push_back({names[7], "Vectorize", {2, 4, 8}, 2});         // bf16 per global load
    v.push_back({names[8], "Unroll", {1, 2}, 1});
    v.push_back({names[9], "Layout", {0, 1}, 0});               // weight stored KxN / NxK
    // tile order: plain / XCD-grouped, m fastest / XCD-grouped over the
    // tiles that hold rows, n fastest
    v.push_back({names[10], "Parallel", {0, 1, 2}, 0});
    v.push_back({names[11], "Parallel", {1, 2}, 1});            // waves per SIMD to budget registers for
}

static const char *const PLAIN[12] = {"tile_m", "tile_n", "tile_k", "waves_m", "waves_n", "mfma",
                                      "stages", "vec", "unroll", "layout", "grid", "occ"};
static const char *const UP[12] = {"up.tile_m", "up.tile_n", "up.tile_k", "up.waves_m",
                                   "up.waves_n", "up.mfma", "up.stages", "up.vec", "up.unroll",
                                   "up.layout", "up.grid", "up.occ"};
static const char *const DOWN[12] = {"down.tile_m", "down.tile_n", "down.tile_k", "down.waves_m",
                                     "down.waves_n", "down.mfma", "down.stages", "down.vec",
                                     "down.unroll", "down.layout", "down.grid", "down.occ"};

static std::vector<KnobDef> mlp_knobs() {
    std::vector<KnobDef> v;
    add_gemm_block(v, UP, {16, 32, 64, 128, 256}, {32, 64, 128});
    add_gemm_block(v, DOWN, {16, 32, 64, 128, 256}, {32, 64, 128});
    v.push_back({"fuse", "ComputeLocation", {0, 1}, 0});
    // the column tiles of a last, partial round of workgroups run as a
    // second launch, so that round is as short as its share of the work:
    // 1 - with half-height tiles (twice as many, half the work each);
    // 2 - with full tiles whose K range is cut in two (fp32 partial sums,
    // added, with the epilogue, by a separate kernel)
    v.push_back({"up.tail", "Parallel", {0, 1, 2}, 0});
    v.push_back({"down.tail", "Parallel", {0, 1, 2}, 0});
    // K range of the down projection cut over 1, 2 or 4 workgroups per
    // output tile (fp32 partial sums, added by a separate kernel)
    v.push_back({"down.split", "Parallel", {1, 2, 4}, 1});
    return v;
}

static std::vector<KnobDef> moe_knobs() {
    std::vector<KnobDef> v = mlp_knobs();
    v.resize(v.size() - 3);     // expert groups are ragged: no tail or K split
    // 1: an expert's last, partial M tile runs a second copy of the GEMM's
    // main loop that skips the fragment reads and MFMAs of its empty row
    // blocks (full tiles keep the first copy unchanged)
    v.push_back({"up.skip", "ComputeLocation", {0, 1}, 0});
    v.push_back({"down.skip", "ComputeLocation", {0, 1}, 0});
    return v;
}

static std::vector<KnobDef> conv_knobs() {
    std::vector<KnobDef> v;
    add_gemm_block(v, PLAIN, {16, 32, 64, 80, 128, 160, 256, 320}, {32, 64, 128});
    v.push_back({"fuse", "ComputeLocation", {0, 1}, 0});
    return v;
}

static std::vector<KnobDef> attention_knobs() {
    return {
        {"block_m", "TileSize", {16, 32, 64, 128, 256}, 16},
        {"block_n", "TileSize", {32, 64, 128}, 32},
        {"waves", "Parallel", {1, 2, 4, 8}, 1},
        {"mfma", "TileSize", {16, 32}, 16},
        {"stages", "ComputeLocation", {1, 2, 3, 4, 5}, 1},
        {"vec", "Vectorize", {2, 4, 8}, 2},
        {"unroll", "Unroll", {1, 2}, 1},
        {"order", "Parallel", {0, 1, 2}, 0},
        {"occ", "Parallel", {1, 2, 4}, 1},
        {"splits", "Parallel", {1, 2, 4}, 1},
        {"chunk", "Parallel", {0, 4, 8, 16}, 0},   // key tiles per work item (0: whole row)
    };
}

const std::vector<KnobDef> &knobs_for(int32_t kind) {
    static const std::vector<KnobDef> empty;
    static const std::vector<KnobDef> g = gemm_f32_knobs();
    static const std::vector<KnobDef> a = attention_knobs();
    static const std::vector<KnobDef> m = mlp_knobs();
    static const std::vector<KnobDef> e = moe_knobs();
    static const std::vector<KnobDef> c = conv_knobs();
    switch (kind) {
        case RC_OP_GEMM_F32: return g;
        case RC_OP_ATTENTION: return a;
        case RC_OP_GATED_MLP: return m;
        case RC_OP_MOE: return e;
        case RC_OP_CONV2D: return c;
        default: return empty;
    }
}

int knob_index(int32_t kind, const char *name) {
    const auto &k = knobs_for(kind);
    for (size_t i = 0; i < k.size(); ++i)
        if (std::strcmp(k[i].name, name) == 0) return (int)i;
    return -1;
}

static int expected_dims(int32_t kind) {
    switch (kind) {
        case RC_OP_GEMM_F32: return 3;
        case RC_OP_ATTENTION: return 4;
        case RC_OP_GATED_MLP: return 3;
        case RC_OP_MOE: return 5;
        case RC_OP_CONV2D: return 8;
        default: return -1;
    }
}

bool desc_ok(const rc_op_desc *d) {
    if (!d || d->struct_size < sizeof(rc_op_desc)) return false;
    int nd = expected_dims(d->kind);
    if (nd < 0) return false;
    for (int i = 0; i < nd; ++i) {
        bool pad = (d->kind == RC_OP_CONV2D && i == 7);
        if (pad ? d->dim[i] < 0 : d->dim[i] <= 0) return false;
    }
    return true;
}

int32_t kv(const rc_op_desc *d, const rc_schedule *s, const char *name) {
    int i = knob_index(d->kind, name);
    return i < 0 ? -1 : s->knob[i];
}

// A tile value v of knob `name` over an extent it need not fill is redundant
// when half of it is also an allowed value and still covers the extent: the
// larger tile only adds empty work.
static bool redundant_tile(const rc_op_desc *d, const char *name, int v, int64_t extent) {
    if (v <= extent || v / 2 < extent) return false;
    const int i = knob_index(d->kind, name);
    if (i < 0) return false;
    for (int32_t a : knobs_for(d->kind)[i].values)
        if (a == v / 2) return true;
    return false;
}

static std::string fmt(const char *f, ...) {
    char buf[256];
    va_list ap;
    va_start(ap, f);
    vsnprintf(buf, sizeof buf, f, ap);
    va_end(ap);
    return buf;
}

static const int64_t LDS_LIMIT = 163840;   // bytes one workgroup may allocate on gfx950

// Depth of the direct-to-LDS ring of bf16 GEMM stages 7: as many stages as
// fit the LDS share of one workgroup when occ waves per SIMD are resident,
// at most 12, and few enough that the loads a wave keeps in flight
// (NSTAGE - 2 tiles) fit the 6-bit vector-memory counter.
int gemm_ring_stages(int tm, int tn, int tk, int nb, int waves, int occ) {
    const int64_t sb = (int64_t)(tm + nb * tn) * tk * 2;
    const int64_t wgs = std::max<int64_t>(1, (occ * 4 + waves - 1) / waves);
    const int64_t lpt = std::max<int64_t>(1, sb / 1024 / waves);
    return (int)std::min<int64_t>(std::min<int64_t>(12, LDS_LIMIT / (wgs * sb)), 63 / lpt + 2);
}

// Column split of a GEMM block whose workgroups end in a partial round:
// the columns of whole rounds stay in the first launch, the rest go to a
// second launch with half-height tiles.  Workgroups per CU are estimated
// from the occupancy the schedule asks for and its LDS.  Returns false
// when every round is full (nothing to split).
bool gemm_tail_split(int tm, int tn, int tk, int nb, int waves, int occ, int st, int64_t M, int64_t N,
                     int64_t *main_cols, int64_t *tail_cols) {
    const int64_t stage_bytes = ((int64_t)tm * tk + (int64_t)nb * tn * tk) * 2;
    int64_t nbuf = st == 4 || st == 6 ? 3 : st > 1 ? 2 : 1;
    if (st == 7) nbuf = gemm_ring_stages(tm, tn, tk, nb, waves, occ);
    const int64_t by_lds = std::max<int64_t>(1, LDS_LIMIT / (nbuf * stage_bytes));
    const int64_t wgs = std::min<int64_t>(by_lds, std::max<int64_t>(1, (int64_t)occ * 4 / waves));
    const int64_t slots = 256 * wgs, ntm = (M + tm - 1) / tm, cols = N / tn;
    const int64_t full_cols = (ntm * cols / slots) * slots / ntm;   // whole rounds, whole columns
    if (full_cols <= 0 || full_cols >= cols) return false;
    *main_cols = full_cols;
    *tail_cols = cols - full_cols;
    return true;
}

// Rules for one bf16 GEMM stage of shape M x N x K (M < 0: ragged expert
// groups), NB weight operands sharing the A tile.  Any M is legal: the last
// M tile's missing rows are predicated off.
static std::string check_bf16_block(const rc_op_desc *d, const rc_schedule *s,
                                    const char *const names[12], int64_t M, int64_t N, int64_t K,
                                    int NB, const char *tag, bool im2col = false) {
    int tm = kv(d, s, names[0]), tn = kv(d, s, names[1]), tk = kv(d, s, names[2]);
    int wm = kv(d, s, names[3]), wn = kv(d, s, names[4]), mf = kv(d, s, names[5]);
    int st = kv(d, s, names[6]), vec = kv(d, s, names[7]), un = kv(d, s, names[8]);
    int lay = kv(d, s, names[9]);
    (void)st;
    int nt = 64 * wm * wn;
    if (tm % wm || (tm / wm) % mf)
        return fmt("%s: tile_m/waves_m = %d/%d is not a multiple of the %dx%d MFMA", tag, tm, wm,
                   mf, mf);
    if (tn % wn || (tn / wn) % mf)
        return fmt("%s: tile_n/waves_n = %d/%d is not a multiple of the %dx%d MFMA", tag, tn, wn,
                   mf, mf);
    if (tk % 32) return fmt("%s: tile_k %d is not a multiple of 32", tag, tk);
    // rows need not fill the last M tile (predicated, for dense and ragged
    // rows alike); a tile twice the rows it covers adds only empty work
    if (M > 0 && redundant_tile(d, names[0], tm, M))
        return fmt("%s: tile_m %d: tile_m %d already covers M = %lld", tag, tm, tm / 2, (long long)M);
    if (N % tn) return fmt("%s: tile_n %d does not divide N = %lld", tag, tn, (long long)N);
    if (K % tk) return fmt("%s: tile_k %d does not divide K = %lld", tag, tk, (long long)K);
    // register-staged loads: every thread moves whole vectors of each tile
    // (the direct-to-LDS stages 4, 6 and 7 have their own wave-load rules)
    const bool dma = st == 4 || st == 6 || st == 7;
    if (!dma && (int64_t)tm * tk % ((int64_t)vec * nt))
        return fmt("%s: A tile %dx%d does not split into %d threads x %d-wide loads", tag, tm, tk,
                   nt, vec);
    if (!dma && (int64_t)tn * tk % ((int64_t)vec * nt))
        return fmt("%s: B tile %dx%d does not split into %d threads x %d-wide loads", tag, tk, tn,
                   nt, vec);
    if (lay == 0 && tn % vec) return fmt("%s: vec %d does not divide tile_n %d", tag, vec, tn);
    if (st == 4) {
        // direct-to-LDS loads: whole 1 KiB wave-loads of 16-byte chunks
        if (lay != 1) return fmt("%s: direct-to-LDS staging needs weights stored N x K", tag);
        if (vec != 8) return fmt("%s: direct-to-LDS staging moves 16-byte vectors (vec 8)", tag);
        if (im2col) return fmt("%s: direct-to-LDS staging cannot zero-fill padded im2col rows", tag);
        if (((int64_t)tm * tk / 512) % (wm * wn) || tm * tk < 512 * wm * wn)
            return fmt("%s: A tile is not a whole number of 1 KiB wave-loads per wave", tag);
        if (((int64_t)tn * tk / 512) % (wm * wn) || tn * tk < 512 * wm * wn)
            return fmt("%s: B tile is not a whole number of 1 KiB wave-loads per wave", tag);
    }
    if (st == 6) {
        // ping-pong: two groups of four waves, one wave of each per SIMD;
        // group 0 moves whole tiles direct to LDS, every wave holds a whole
        // K tile of fragments in registers
        if (wm * wn != 8) return fmt("%s: ping-pong staging needs 8 waves (has %d)", tag, wm * wn);
        if (lay != 1) return fmt("%s: ping-pong staging needs weights stored N x K", tag);
        if (vec != 8) return fmt("%s: ping-pong staging moves 16-byte vectors (vec 8)", tag);
        if (im2col) return fmt("%s: ping-pong staging cannot zero-fill padded im2col rows", tag);
        if (((int64_t)tm * tk / 512) % 4 || tm * tk < 512 * 4)
            return fmt("%s: A tile is not a whole number of 1 KiB wave-loads per loading wave", tag);
        if (((int64_t)tn * tk / 512) % 4 || tn * tk < 512 * 4)
            return fmt("%s: B tile is not a whole number of 1 KiB wave-loads per loading wave", tag);
        if (((int64_t)tm * tk + (int64_t)NB * tn * tk) / 512 / 4 > 62)
            return fmt("%s: loads per loading wave per K tile exceed the 6-bit vector-memory counter", tag);
        if (kv(d, s, names[11]) != 2) return fmt("%s: ping-pong staging runs two waves per SIMD (occ 2)", tag);
        int64_t frag = (int64_t)(tm / wm / mf + NB * (tn / wn / mf)) * (tk / (mf == 16 ? 32 : 16)) * 4;
        int64_t accr = (int64_t)NB * tm * tn / nt;
        if (accr + frag > 224)
            return fmt("%s: %lld accumulator + %lld fragment registers per lane exceed 224", tag,
                       (long long)accr, (long long)frag);
    }
    if (st == 7) {
        // deep direct-to-LDS ring of buffer loads (range-checked, so
        // padded im2col taps and missing rows load zeros)
        if (lay != 1) return fmt("%s: the direct-to-LDS ring needs weights stored N x K", tag);
        if (vec != 8) return fmt("%s: the direct-to-LDS ring moves 16-byte vectors (vec 8)", tag);
        if (((int64_t)tm * tk / 512) % (wm * wn) || tm * tk < 512 * wm * wn)
            return fmt("%s: A tile is not a whole number of 1 KiB wave-loads per wave", tag);
        if (((int64_t)tn * tk / 512) % (wm * wn) || tn * tk < 512 * wm * wn)
            return fmt("%s: B tile is not a whole number of 1 KiB wave-loads per wave", tag);
        // 32-bit buffer offsets, and an out-of-range offset (2^31) past every operand
        if ((M > 0 ? M : 0) * K * 2 >= (1LL << 31) || N * K * 2 >= (1LL << 31))
            return fmt("%s: operands of 2 GiB or more exceed the ring's 32-bit buffer offsets", tag);
        const int ns = gemm_ring_stages(tm, tn, tk, NB, wm * wn, kv(d, s, names[11]));
        if (ns < 3) return fmt("%s: the LDS holds %d ring stages of this tile (needs 3)", tag, ns);
        const int64_t lpt = ((int64_t)tm * tk + (int64_t)NB * tn * tk) / 512 / (wm * wn);
        if ((ns - 2) * lpt > 63)
            return fmt("%s: %lld loads per wave in flight exceed the 6-bit vector-memory counter", tag,
                       (long long)((ns - 2) * lpt));
        const int64_t frag = (int64_t)(tm / wm / mf + NB * (tn / wn / mf)) * 4 * 2;
        const int64_t accr = (int64_t)NB * tm * tn / nt;
        if (accr + frag > 448)
            return fmt("%s: %lld accumulator + %lld fragment registers per lane exceed 448", tag,
                       (long long)accr, (long long)frag);
    }
    const int64_t stage_bytes = ((int64_t)tm * tk + (int64_t)NB * tn * tk) * 2;
    int64_t lds = (int64_t)(st == 4 || st == 6 ? 3 : st > 1 ? 2 : 1) * stage_bytes;
    if (st == 7) lds = (int64_t)gemm_ring_stages(tm, tn, tk, NB, wm * wn, kv(d, s, names[11])) * stage_bytes;
    if (lds > LDS_LIMIT)
        return fmt("%s: LDS %lld B exceeds %lld B", tag, (long long)lds, (long long)LDS_LIMIT);
    int64_t acc = (int64_t)NB * tm * tn / nt;
    if (acc > 256) return fmt("%s: %lld accumulators per lane exceed 256", tag, (long long)acc);
    int occ = kv(d, s, names[11]);
    if (occ > 1) {
        // occ waves per SIMD: the registers of occ waves share 512 per lane,
        // and enough workgroups must fit in the CU's LDS.
        if (acc > 512 / occ - 32) return fmt("%s: %lld accumulators leave no registers at %d waves/SIMD", tag, (long long)acc, occ);
        int64_t waves = (int64_t)wm * wn, wgs = (occ * 4 + waves - 1) / waves;
        if (wgs * lds > LDS_LIMIT) return fmt("%s: %lld workgroups of %lld B LDS do not fit a CU", tag, (long long)wgs, (long long)lds);
    }
    // register staging: one set of the next tile (stages 2, 3), two (5)
    int64_t stage_regs = (st == 2 || st == 3 || st == 5) ? ((int64_t)tm * tk + (int64_t)NB * tn * tk) / (2 * nt) : 0;
    if (st == 5) stage_regs *= 2;
    if (acc + stage_regs > 384)
        return fmt("%s: %lld accumulator + %lld staging registers per lane exceed 384", tag,
                   (long long)acc, (long long)stage_regs);
    if ((K / tk) % un) return fmt("%s: unroll %d does not divide %lld K tiles", tag, un,
                                  (long long)(K / tk));
    return "";
}

std::string check_schedule(const rc_op_desc *d, const rc_schedule *s) {
    const auto &kt = knobs_for(d->kind);
    if (s->struct_size < sizeof(rc_schedule)) return "schedule struct_size too small";
    if (s->nknobs != (int32_t)kt.size()) return fmt("schedule has %d knobs, operator has %d",
                                                    s->nknobs, (int)kt.size());
    for (size_t i = 0; i < kt.size(); ++i) {
        bool found = false;
        for (int32_t v : kt[i].values) found |= (v == s->knob[i]);
        if (!found) return fmt("knob %s = %d is not an allowed value", kt[i].name, s->knob[i]);
    }
    const int64_t *D = d->dim;
    switch (d->kind) {
        case RC_OP_GEMM_F32: {
            int tm = kv(d, s, "tile_m"), tn = kv(d, s, "tile_n"), tk = kv(d, s, "tile_k");
            int wm = kv(d, s, "waves_m"), wn = kv(d, s, "waves_n"), vec = kv(d, s, "vec");
            int st = kv(d, s, "stages"), un = kv(d, s, "unroll"), lay = kv(d, s, "layout");
            int64_t M = D[0], N = D[1], K = D[2];
            int nt = 64 * wm * wn;
            int sp = kv(d, s, "splits");
            if (st == 3) {
                // streaming: one 16-row MFMA block of outputs (decode-shaped
                // operators), 64 columns per workgroup as 16 lanes x 4
                // floats, B stored [K][N]; the waves and the SPLITS
                // workgroups of a column tile each take whole batches of
                // tile_k rows (16-row blocks) of the K range
                if (M > 16) return fmt("streaming stage needs M <= 16 (one MFMA row block), M = %lld", (long long)M);
                if (tm != 16) return "streaming stage takes tile_m 16";
                if (tn != 64) return "streaming stage takes tile_n 64 (16 lanes x 4 floats)";
                if (vec != 4) return "streaming stage moves 16-byte vectors (vec 4)";
                if (lay != 0) return "streaming stage reads B stored K x N";
                if (tk % 16) return fmt("streaming stage takes tile_k in 16-row blocks (tile_k %d)", tk);
                if (N % tn) return fmt("tile_n %d does not divide N = %lld", tn, (long long)N);
                int64_t per = (int64_t)sp * wm * wn * tk;
                if (K % per)
                    return fmt("K = %lld is not a whole number of %d-row batches for %d splits x %d waves",
                               (long long)K, tk, sp, wm * wn);
                // unroll sets the prefetch depth: min(2 x unroll, batches
                // per wave) batches of tile_k rows (5 tile_k / 4 registers
                // each) in flight
                int64_t nb = K / per;
                if (un > 1 && un >= nb)
                    return fmt("unroll %d: all %lld batches per wave are already in flight at a smaller unroll", un,
                               (long long)nb);
                int64_t pf = std::min<int64_t>(2 * un, nb);
                if (pf * tk * 5 / 4 > 160)
                    return fmt("%lld batches of %d rows in flight need more than 160 registers", (long long)pf, tk);
                return "";
            }
            if (sp != 1) return "K splits across workgroups need the streaming stage (stages 3)";
            if ((tm / wm) % 16 || tm % wm) return fmt("tile_m/waves_m = %d/%d is not a multiple of 16", tm, wm);
            if ((tn / wn) % 16 || tn % wn) return fmt("tile_n/waves_n = %d/%d is not a multiple of 16", tn, wn);
            // tiles may cross the edges of M, N and K (zero-filled loads,
            // predicated stores), but a tile twice the extent it covers adds
            // only empty work (the halved tile covers it too); a vector load
            // must not cross a row end
            if (redundant_tile(d, "tile_m", tm, M)) return fmt("tile_m %d: tile_m %d already covers M = %lld", tm, tm / 2, (long long)M);
            if (redundant_tile(d, "tile_n", tn, N)) return fmt("tile_n %d: tile_n %d already covers N = %lld", tn, tn / 2, (long long)N);
            if (redundant_tile(d, "tile_k", tk, K)) return fmt("tile_k %d: tile_k %d already covers K = %lld", tk, tk / 2, (long long)K);
            if (K % vec) return fmt("vec %d does not divide the rows of A (K = %lld)", vec, (long long)K);
            if (lay == 0 && N % vec) return fmt("vec %d does not divide the rows of B (N = %lld)", vec, (long long)N);
            if ((tm * tk) % (vec * nt))
                return fmt("A tile %dx%d does not split into %d threads x %d-wide loads", tm, tk, nt, vec);
            if ((tk * tn) % (vec * nt))
                return fmt("B tile %dx%d does not split into %d threads x %d-wide loads", tk, tn, nt, vec);
            if (tk % vec) return fmt("vec %d does not divide tile_k %d", vec, tk);
            if (lay == 0 && tn % vec) return fmt("vec %d does not divide tile_n %d", vec, tn);
            const int64_t ktiles = (K + tk - 1) / tk;
            if (ktiles % un) return fmt("unroll %d does not divide the %lld K tiles", un, (long long)ktiles);
            int64_t lds = (int64_t)st * (tm * (tk + 1) + tk * (tn + 1)) * 4;
            if (lds > LDS_LIMIT) return fmt("LDS %lld B exceeds limit", (long long)lds);
            return "";
        }
        case RC_OP_ATTENTION: {
            int bm = kv(d, s, "block_m"), bn = kv(d, s, "block_n"), w = kv(d, s, "waves");
            int mf = kv(d, s, "mfma"), st = kv(d, s, "stages");
            int64_t S = D[2], Dh = D[3];
            if (bm % w) return fmt("block_m %d is not divisible by waves %d", bm, w);
            int rpw = bm / w;
            if (rpw % mf) return fmt("rows per wave %d is not a multiple of the %dx%d MFMA", rpw, mf, mf);
            if (rpw / mf > 2) return fmt("rows per wave %d exceeds two MFMA blocks", rpw);
            if (bn % 32) return fmt("block_n %d is not a multiple of 32", bn);
            // the sequence need not fill the last query or key tile (rows
            // past it are clamped on load, masked and not stored), but a
            // block twice the sequence adds only empty work
            if (redundant_tile(d, "block_m", bm, S)) return fmt("block_m %d: block_m %d already covers S = %lld", bm, bm / 2, (long long)S);
            if (redundant_tile(d, "block_n", bn, S)) return fmt("block_n %d: block_n %d already covers S = %lld", bn, bn / 2, (long long)S);
            // the K tile's LDS swizzle XORs 16-byte chunk indices, so a row
            // must hold a power-of-two number of chunks
            if (Dh != 32 && Dh != 64 && Dh != 128 && Dh != 256)
                return fmt("head dim %lld must be 32, 64, 128 or 256", (long long)Dh);
            int sp = kv(d, s, "splits");
            if (w * sp > 16) return fmt("waves x splits = %d exceeds 16 waves per workgroup", w * sp);
            if (st >= 4) {
                // direct-to-LDS ring: whole 1 KiB wave-loads, key-major V read
                // by the 16x16 transposing load
                if (mf != 16) return "direct-to-LDS attention uses the 16x16 MFMA shape";
                if (kv(d, s, "vec") != 8) return "direct-to-LDS loads move 16-byte vectors (vec 8)";
                if ((bn * Dh / 512) % w || bn * Dh < 512 * w)
                    return fmt("K/V tile of %d x %lld is not a whole number of 1 KiB wave-loads per wave", bn, (long long)Dh);
                if (2 * bn * Dh / 512 / w > 62)
                    return fmt("%lld loads per wave per K/V tile exceed the 6-bit vector-memory counter", (long long)(2 * bn * Dh / 512 / w));
            }
            // K tile + padded V^T tile per stage and split (for the
            // direct-to-LDS ring: three K/V slots, two per split, or four per
            // split with the pipelined stages 5)
            int64_t vts = bn + (mf == 16 ? 16 : 8);   // padded V^T row
            int64_t lds = st >= 4 ? (st == 5 ? 4 * sp : sp > 1 ? 2 * sp : 3) * 2 * (int64_t)bn * Dh * 2
                                  : (int64_t)sp * (st > 1 ? 2 : 1) * ((int64_t)bn * Dh + Dh * vts) * 2;
            if (lds > LDS_LIMIT) return fmt("LDS %lld B exceeds limit", (long long)lds);
            int64_t mf_acc = (mf == 16) ? 4 : 16;
            int64_t merge = (int64_t)(sp - 1) * w * ((rpw / mf) * 2 * mf + (rpw / mf) * (Dh / mf) * mf_acc * 64) * 4;
            if (merge > lds) return fmt("merging %d splits needs %lld B of LDS, more than the %lld B tiles", sp, (long long)merge, (long long)lds);
            int64_t regs = (int64_t)rpw * Dh / 64 + (int64_t)bn * rpw / 64 + (int64_t)rpw * Dh / 128;
            if (regs > 320) return fmt("%lld registers per lane for O, S and Q exceed 320", (long long)regs);
            int occ = kv(d, s, "occ");
            if (occ > 1) {
                if (regs > 512 / occ - 64)
                    return fmt("%lld registers per lane for O, S and Q leave too few at %d waves/SIMD", (long long)regs, occ);
                int64_t wgs = (occ * 4 + w * sp - 1) / (w * sp);
                if (wgs * lds > LDS_LIMIT)
                    return fmt("%lld workgroups of %lld B LDS do not fit a CU", (long long)wgs, (long long)lds);
            }
            int ch = kv(d, s, "chunk");
            if (ch > 0 && ch >= (S + bn - 1) / bn)
                return fmt("chunk of %d key tiles covers all %lld key tiles (same as chunk 0)", ch,
                           (long long)((S + bn - 1) / bn));
            if (kv(d, s, "order") == 2 && ((S + bm - 1) / bm) % 2)
                return "paired tile order needs an even number of query tiles";
            return "";
        }
        case RC_OP_GATED_MLP: {
            int64_t T = D[0], Hd = D[1], I = D[2];
            std::string r = check_bf16_block(d, s, UP, T, I, Hd, 2, "up");
            if (!r.empty()) return r;
            r = check_bf16_block(d, s, DOWN, T, Hd, I, 1, "down");
            if (!r.empty()) return r;
            for (int b = 0; b < 2; ++b) {
                const char *const *nm = b == 0 ? UP : DOWN;
                const char *tag = b == 0 ? "up" : "down";
                const int tmode = kv(d, s, b == 0 ? "up.tail" : "down.tail");
                if (tmode == 0) continue;
                const int64_t N = b == 0 ? I : Hd, K = b == 0 ? Hd : I;
                const int nb = b == 0 ? 2 : 1;
                int64_t mc = 0, tc = 0;
                if (!gemm_tail_split(kv(d, s, nm[0]), kv(d, s, nm[1]), kv(d, s, nm[2]), nb,
                                     kv(d, s, nm[3]) * kv(d, s, nm[4]), kv(d, s, nm[11]), kv(d, s, nm[6]), T, N,
                                     &mc, &tc))
                    return fmt("%s: tail split: no partial round of workgroups to split", tag);
                if (tmode == 2) {
                    // full tiles, K range cut in two; the gate/up epilogue
                    // moves into the summing kernel
                    const int tk = kv(d, s, nm[2]), un = kv(d, s, nm[8]);
                    if (b == 0 && kv(d, s, "fuse") != 1)
                        return "up: a K-split tail needs the fused SwiGLU epilogue (fuse 1)";
                    if (K % (2LL * tk))
                        return fmt("%s: K-split tail: K = %lld is not a whole number of %d-wide K tiles per half", tag, (long long)K, tk);
                    if ((K / tk / 2) % un)
                        return fmt("%s: K-split tail: unroll %d does not divide the %lld K tiles of a half", tag, un, (long long)(K / tk / 2));
                    continue;
                }
                // the tail launch runs the same schedule with half-height tiles
                rc_schedule h = *s;
                h.knob[knob_index(d->kind, nm[0])] = kv(d, s, nm[0]) / 2;
                std::string why = check_bf16_block(d, &h, nm, T, N, K, nb, tag);
                if (!why.empty()) return fmt("%s: tail split: the half-height tile is illegal (%s)", tag, why.c_str());
            }
            const int sk = kv(d, s, "down.split");
            if (sk > 1) {
                const int tk = kv(d, s, "down.tile_k"), un = kv(d, s, "down.unroll");
                if (kv(d, s, "down.tail") != 0) return "down: the tail split and the K split do not combine";
                if (I % ((int64_t)sk * tk))
                    return fmt("down: K = %lld is not a whole number of %d-wide K tiles per split of %d", (long long)I, tk, sk);
                if ((I / tk / sk) % un)
                    return fmt("down: unroll %d does not divide the %lld K tiles of a split", un, (long long)(I / tk / sk));
            }
            return "";
        }
        case RC_OP_MOE: {
            int64_t Hd = D[1], E = D[2], I = D[3], topk = D[4];
            if (topk > E) return "topk exceeds the number of experts";
            // the routing kernel (one workgroup of 1024 threads) keeps one
            // thread per expert and per-wave row counts of every expert in
            // LDS (16 x E x 4 B)
            if (E > 1024) return fmt("%lld experts exceed the routing kernel's 1024", (long long)E);
            if (D[0] * topk > INT32_MAX / 2) return "routed rows exceed the 32-bit row indices";
            if ((kv(d, s, "up.stages") == 7 || kv(d, s, "down.stages") == 7) &&
                std::max(D[0] * Hd, D[0] * topk * I) * 2 >= (1LL << 31))
                return "activations of 2 GiB or more exceed the ring's 32-bit buffer offsets";
            // the ping-pong stage has no partial-tile copy of its loop: a skip
            // there would only duplicate the schedule without it
            if (kv(d, s, "up.skip") == 1 && kv(d, s, "up.stages") == 6)
                return "up: the ping-pong stage (6) has no partial-tile loop to skip rows in";
            if (kv(d, s, "down.skip") == 1 && kv(d, s, "down.stages") == 6)
                return "down: the ping-pong stage (6) has no partial-tile loop to skip rows in";
            std::string r = check_bf16_block(d, s, UP, -1, I, Hd, 2, "up");
            if (!r.empty()) return r;
            return check_bf16_block(d, s, DOWN, -1, Hd, I, 1, "down");
        }
        case RC_OP_CONV2D: {
            int64_t N = D[0], H = D[1], W = D[2], C = D[3], K = D[4], R = D[5], S = D[6], pad = D[7];
            int64_t P = H + 2 * pad - R + 1, Q = W + 2 * pad - S + 1;
            if (P <= 0 || Q <= 0) return "empty output";
            int tk = kv(d, s, "tile_k");
            if (C % tk) return fmt("tile_k %d does not divide C = %lld (a K tile must stay in one filter tap)", tk, (long long)C);
            if (R * S > 32) return fmt("%lld filter taps exceed the 32-bit tap mask", (long long)(R * S));
            return check_bf16_block(d, s, PLAIN, N * P * Q, K, R * S * C, 1, "conv", true);
        }
    }
    return "unknown operator kind";
}

}  // namespace rc

using namespace rc;

extern "C" {

const char *rc_status_str(rc_status s) {
    switch (s) {
        case RC_OK: return "RC_OK";
        case RC_ERR_INVALID_ARGUMENT: return "RC_ERR_INVALID_ARGUMENT";
        case RC_ERR_ILLEGAL_SCHEDULE: return "RC_ERR_ILLEGAL_SCHEDULE";
        case RC_ERR_UNSUPPORTED: return "RC_ERR_UNSUPPORTED";
        case RC_ERR_COMPILE: return "RC_ERR_COMPILE";
        case RC_ERR_HIP: return "RC_ERR_HIP";
        case RC_ERR_OUT_OF_MEMORY: return "RC_ERR_OUT_OF_MEMORY";
        case RC_ERR_MISALIGNED: return "RC_ERR_MISALIGNED";
        case RC_ERR_BUDGET: return "RC_ERR_BUDGET";
    }
    return "RC_ERR_UNKNOWN";
}

const char *rc_last_error(void) { return g_err.c_str(); }

rc_status rc_op_init(rc_op_desc *d, int32_t kind, const int64_t *dims, int32_t ndims,
                     int32_t flags) {
    if (!d || !dims) return fail(RC_ERR_INVALID_ARGUMENT, "null descriptor or dims");
    int nd = expected_dims(kind);
    if (nd < 0) return fail(RC_ERR_UNSUPPORTED, "unknown operator kind");
    if (ndims != nd) return fail(RC_ERR_INVALID_ARGUMENT, fmt("kind %d takes %d dims, got %d", kind, nd, ndims));
    rc_op_desc t;
    std::memset(&t, 0, sizeof t);
    t.struct_size = sizeof(rc_op_desc);
    t.kind = kind;
    for (int i = 0; i < nd; ++i) t.dim[i] = dims[i];
    t.flags = flags;
    if (!desc_ok(&t)) return fail(RC_ERR_INVALID_ARGUMENT, "dimensions must be positive");
    const int32_t allowed = kind == RC_OP_ATTENTION ? RC_FLAG_CAUSAL : kind == RC_OP_CONV2D ? RC_FLAG_NO_ACT : 0;
    if (flags & ~allowed) return fail(RC_ERR_INVALID_ARGUMENT, fmt("flags 0x%x not defined for kind %d", flags, kind));
    if (kind == RC_OP_MOE && t.dim[4] > t.dim[2])
        return fail(RC_ERR_INVALID_ARGUMENT, "topk exceeds the number of experts");
    *d = t;
    clear_error();
    return RC_OK;
}

double rc_op_flops(const rc_op_desc *d) {
    if (!desc_ok(d)) return -1.0;
    const int64_t *D = d->dim;
    switch (d->kind) {
        case RC_OP_GEMM_F32: return 2.0 * D[0] * D[1] * D[2];
        case RC_OP_ATTENTION: {
            double S = (double)D[2];
            double pairs = (d->flags & RC_FLAG_CAUSAL) ? S * (S + 1) / 2 : S * S;
            return 4.0 * D[3] * D[0] * D[1] * pairs;
        }
        case RC_OP_GATED_MLP: return 6.0 * D[0] * D[1] * D[2];
        case RC_OP_MOE: return 6.0 * D[0] * D[4] * D[1] * D[3];
        case RC_OP_CONV2D: {
            double P = D[1] + 2 * D[7] - D[5] + 1, Q = D[2] + 2 * D[7] - D[6] + 1;
            return 2.0 * D[0] * P * Q * D[4] * D[5] * D[6] * D[3];
        }
    }
    return -1.0;
}

double rc_op_bytes(const rc_op_desc *d) {
    if (!desc_ok(d)) return -1.0;
    const int64_t *D = d->dim;
    switch (d->kind) {
        case RC_OP_GEMM_F32: return 4.0 * (D[0] * D[2] + D[2] * D[1] + D[0] * D[1]);
        case RC_OP_ATTENTION: return 2.0 * 4 * D[0] * D[1] * D[2] * D[3];
        case RC_OP_GATED_MLP: return 2.0 * (2 * D[0] * D[1] + 3 * D[1] * D[2]);
        case RC_OP_MOE:
            return 2.0 * (2 * D[0] * D[1] + 3 * D[2] * D[1] * D[3]) + 8.0 * D[0] * D[4];
        case RC_OP_CONV2D: {
            double P = D[1] + 2 * D[7] - D[5] + 1, Q = D[2] + 2 * D[7] - D[6] + 1;
            return 2.0 * D[0] * D[1] * D[2] * D[3] + 2.0 * D[4] * D[5] * D[6] * D[3] + 4.0 * D[4] +
                   2.0 * D[0] * P * Q * D[4];
        }
    }
    return -1.0;
}

double rc_peak_flops(const rc_op_desc *d) {
    if (!desc_ok(d)) return -1.0;
    return d->kind == RC_OP_GEMM_F32 ? 157.3e12 : 2516.6e12;
}

double rc_peak_bytes_per_s(void) { return 8.0e12; }

int32_t rc_knob_count(const rc_op_desc *d) {
    if (!desc_ok(d)) return -1;
    return (int32_t)knobs_for(d->kind).size();
}

const char *rc_knob_name(const rc_op_desc *d, int32_t knob) {
    if (!desc_ok(d)) return nullptr;
    const auto &k = knobs_for(d->kind);
    return (knob >= 0 && knob < (int32_t)k.size()) ? k[knob].name : nullptr;
}

const char *rc_knob_class(const rc_op_desc *d, int32_t knob) {
    if (!desc_ok(d)) return nullptr;
    const auto &k = knobs_for(d->kind);
    return (knob >= 0 && knob < (int32_t)k.size()) ? k[knob].xform : nullptr;
}

rc_status rc_knob_values(const rc_op_desc *d, int32_t knob, int32_t *vals, int32_t cap,
                         int32_t *n) {
    if (!desc_ok(d) || !n) return fail(RC_ERR_INVALID_ARGUMENT, "bad descriptor");
    const auto &k = knobs_for(d->kind);
    if (knob < 0 || knob >= (int32_t)k.size()) return fail(RC_ERR_INVALID_ARGUMENT, "bad knob");
    *n = (int32_t)k[knob].values.size();
    for (int32_t i = 0; i < *n && i < cap && vals; ++i) vals[i] = k[knob].values[i];
    return RC_OK;
}

rc_status rc_default_schedule(const rc_op_desc *d, rc_schedule *out) {
    if (!desc_ok(d) || !out) return fail(RC_ERR_INVALID_ARGUMENT, "bad descriptor");
    rc_schedule s;
    std::memset(&s, 0, sizeof s);
    s.struct_size = sizeof(rc_schedule);
    const auto &k = knobs_for(d->kind);
    s.nknobs = (int32_t)k.size();
    for (size_t i = 0; i < k.size(); ++i) s.knob[i] = k[i].def;
    std::string why = check_schedule(d, &s);
    if (!why.empty()) return fail(RC_ERR_UNSUPPORTED, "operator shape admits no default schedule: " + why);
    *out = s;
    return RC_OK;
}

rc_status rc_validate(const rc_op_desc *d, const rc_schedule *s, char *why, size_t why_len) {
    if (!desc_ok(d) || !s) return fail(RC_ERR_INVALID_ARGUMENT, "bad descriptor or schedule");
    std::string r = check_schedule(d, s);
    if (why && why_len) {
        std::strncpy(why, r.c_str(), why_len - 1);
        why[why_len - 1] = 0;
    }
    if (!r.empty()) return fail(RC_ERR_ILLEGAL_SCHEDULE, r);
    return RC_OK;
}

rc_status rc_apply(const rc_op_desc *d, const rc_schedule *in, const rc_transform *t,
                   rc_schedule *out) {
    if (!desc_ok(d) || !in || !t || !out) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    if (t->knob < 0 || t->knob >= in->nknobs || in->nknobs > RC_MAX_KNOBS)
        return fail(RC_ERR_INVALID_ARGUMENT, "knob index out of range");
    rc_schedule s = *in;
    s.knob[t->knob] = t->value;
    std::string r = check_schedule(d, &s);
    if (!r.empty()) return fail(RC_ERR_ILLEGAL_SCHEDULE, r);
    *out = s;
    return RC_OK;
}

rc_status rc_enumerate(const rc_op_desc *d, const rc_schedule *at, rc_transform *buf, size_t cap,
                       size_t *n) {
    if (!desc_ok(d) || !at || !n) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    const auto &k = knobs_for(d->kind);
    if (at->nknobs != (int32_t)k.size()) return fail(RC_ERR_INVALID_ARGUMENT, "knob count mismatch");
    size_t cnt = 0;
    for (size_t i = 0; i < k.size(); ++i) {
        for (int32_t v : k[i].values) {
            if (v == at->knob[i]) continue;
            rc_schedule s = *at;
            s.knob[i] = v;
            if (!check_schedule(d, &s).empty()) continue;
            if (buf && cnt < cap) buf[cnt] = rc_transform{(int32_t)i, v};
            ++cnt;
        }
    }
    *n = cnt;
    return RC_OK;
}

rc_status rc_parse_transform(const rc_op_desc *d, const char *text, rc_transform *out) {
    if (!desc_ok(d) || !text || !out) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    // Form: Class(knob=value), whitespace tolerated.
    std::string s;
    for (const char *p = text; *p; ++p)
        if (*p != ' ' && *p != '\t' && *p != '\n' && *p != '\r') s += *p;
    size_t lp = s.find('('), eq = s.find('='), rp = s.find(')');
    if (lp == std::string::npos || eq == std::string::npos || rp == std::string::npos || !(lp < eq && eq < rp) ||
        rp != s.size() - 1)
        return fail(RC_ERR_INVALID_ARGUMENT, "expected Class(knob=value)");
    std::string cls = s.substr(0, lp), name = s.substr(lp + 1, eq - lp - 1),
                val = s.substr(eq + 1, rp - eq - 1);
    int ki = knob_index(d->kind, name.c_str());
    if (ki < 0) return fail(RC_ERR_INVALID_ARGUMENT, "unknown knob " + name);
    const KnobDef &kd = knobs_for(d->kind)[ki];
    if (cls != kd.xform) return fail(RC_ERR_INVALID_ARGUMENT, "knob " + name + " is not a " + cls + " knob");
    if (val.empty()) return fail(RC_ERR_INVALID_ARGUMENT, "missing value");
    char *end = nullptr;
    long v = std::strtol(val.c_str(), &end, 10);
    if (*end) return fail(RC_ERR_INVALID_ARGUMENT, "value is not an integer");
    bool allowed = false;
    for (int32_t a : kd.values) allowed |= (a == v);
    if (!allowed) return fail(RC_ERR_INVALID_ARGUMENT, "value not allowed for " + name);
    *out = rc_transform{ki, (int32_t)v};
    return RC_OK;
}

rc_status rc_schedule_to_string(const rc_op_desc *d, const rc_schedule *s, char *buf, size_t len) {
    if (!desc_ok(d) || !s || !buf || !len) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    const auto &k = knobs_for(d->kind);
    if (s->nknobs != (int32_t)k.size()) return fail(RC_ERR_INVALID_ARGUMENT, "knob count mismatch");
    std::string r;
    for (size_t i = 0; i < k.size(); ++i) {
        if (i) r += ',';
        r += k[i].name;
        r += '=';
        r += std::to_string(s->knob[i]);
    }
    if (r.size() + 1 > len) return fail(RC_ERR_INVALID_ARGUMENT, "buffer too small");
    std::memcpy(buf, r.c_str(), r.size() + 1);
    return RC_OK;
}

rc_status rc_schedule_from_string(const rc_op_desc *d, const char *text, rc_schedule *out) {
    if (!desc_ok(d) || !text || !out) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    rc_schedule s;
    std::memset(&s, 0, sizeof s);
    s.struct_size = sizeof s;
    const auto &k = knobs_for(d->kind);
    s.nknobs = (int32_t)k.size();
    for (size_t i = 0; i < k.size(); ++i) s.knob[i] = k[i].def;
    std::string t(text);
    size_t pos = 0;
    while (pos < t.size()) {
        size_t comma = t.find(',', pos);
        if (comma == std::string::npos) comma = t.size();
        std::string item = t.substr(pos, comma - pos);
        pos = comma + 1;
        if (item.empty()) continue;
        size_t eq = item.find('=');
        if (eq == std::string::npos) return fail(RC_ERR_INVALID_ARGUMENT, "expected name=value");
        int ki = knob_index(d->kind, item.substr(0, eq).c_str());
        if (ki < 0) return fail(RC_ERR_INVALID_ARGUMENT, "unknown knob " + item.substr(0, eq));
        char *end = nullptr;
        long v = std::strtol(item.c_str() + eq + 1, &end, 10);
        if (*end || end == item.c_str() + eq + 1) return fail(RC_ERR_INVALID_ARGUMENT, "bad value in " + item);
        s.knob[ki] = (int32_t)v;
    }
    *out = s;
    return RC_OK;
}

uint64_t rc_schedule_hash(const rc_schedule *s) {
    if (!s) return 0;
    uint64_t h = 1469598103934665603ULL;   // FNV-1a over the knob values
    for (int32_t i = 0; i < s->nknobs && i < RC_MAX_KNOBS; ++i) {
        uint32_t v = (uint32_t)s->knob[i];
        for (int b = 0; b < 4; ++b) {
            h ^= (v >> (8 * b)) & 0xFF;
            h *= 1099511628211ULL;
        }
    }
    return h;
}

}  // extern "C"
