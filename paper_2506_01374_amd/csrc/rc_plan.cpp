// Plans: source generation for a schedule, hipRTC compilation with an
// on-disk code-object cache, module loading, launch and event timing.
#include <dlfcn.h>
#include <hip/hip_runtime_api.h>
#include <hip/hiprtc.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <functional>
#include <map>
#include <memory>
#include <mutex>
#include <sstream>
#include <string>
#include <thread>
#include <vector>

#include "rc_internal.h"

namespace rc {
#include "kernels_src.inc"   // generated: kernel sources as string literals
}

using namespace rc;

namespace {

// ---------------------------------------------------------------------
// Kernel argument blocks; each mirrors the struct its kernel takes by value.
// ---------------------------------------------------------------------
struct GemmF32Args {
    const void *A, *B;
    void *C;
    void *P;   // per-split partial sums (streaming stage with K splits)
};
struct GemmBf16Args {
    const void *A, *B0, *B1;
    void *C, *C1;
    const void *bias, *perm, *offsets, *tile_start;
};
struct EwArgs {
    const void *G, *U, *bias;
    void *out;
};
struct MoeHistArgs {
    const void *ids;
    void *counts;
};
struct MoePrepArgs {
    const void *ids, *counts;
    void *offsets, *perm, *pos, *tile_up, *tile_down;
};
struct MoeCombineArgs {
    const void *Y, *pos, *w;
    void *out;
};
struct AttnArgs {
    const void *Q, *K, *V;
    void *O;
    void *P;   // partial states of query tiles cut into several work items
};

// A kernel's by-value argument block (fixed storage: launching allocates
// nothing on the host).
struct ArgBlob {
    alignas(16) char data[128];
    size_t size = 0;
};

struct Source {
    const char *file;     // kernel source text
    const char *entry;    // kernel function name
    std::string defines;  // generated prologue
};

std::mutex g_mu;
std::string g_cache_dir;
std::map<std::string, hipModule_t> g_modules;   // cache-key -> loaded module

uint64_t fnv1a(const std::string &s, uint64_t h = 1469598103934665603ULL) {
    for (unsigned char c : s) {
        h ^= c;
        h *= 1099511628211ULL;
    }
    return h;
}

std::string lib_dir() {
    Dl_info info;
    if (dladdr((void *)&fnv1a, &info) && info.dli_fname) {
        std::string p(info.dli_fname);
        size_t k = p.rfind('/');
        if (k != std::string::npos) return p.substr(0, k);
    }
    return ".";
}

const std::vector<std::string> &compile_options() {
    static const std::vector<std::string> opts = {
        "--offload-arch=gfx950", "-O3", "-std=c++17",
        // keep the compiler from forming packed fp32 instructions
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"};
    return opts;
}

std::string full_source(const Source &s) { return s.defines + "\n" + s.file; }

std::string cache_key(const Source &s) {
    std::string k = full_source(s);
    for (auto &o : compile_options()) k += "\x1f" + o;
    int maj = 0, min = 0;
    hiprtcVersion(&maj, &min);
    k += "\x1fhiprtc" + std::to_string(maj) + "." + std::to_string(min);
    // the compiler behind hipRTC is identified by the library actually loaded
    Dl_info info;
    if (dladdr((void *)&hiprtcCompileProgram, &info) && info.dli_fname) k += "\x1f" + std::string(info.dli_fname);
    char hex[32];
    snprintf(hex, sizeof hex, "%016llx", (unsigned long long)fnv1a(k));
    return std::string(s.entry) + "_" + hex;
}

bool read_file(const std::string &path, std::vector<char> &out) {
    std::ifstream f(path, std::ios::binary);
    if (!f) return false;
    out.assign(std::istreambuf_iterator<char>(f), std::istreambuf_iterator<char>());
    return !out.empty();
}

void mkdirs(const std::string &dir) {
    std::string cur;
    for (size_t i = 0; i < dir.size(); ++i) {
        cur += dir[i];
        if (dir[i] == '/' || i + 1 == dir.size()) mkdir(cur.c_str(), 0755);
    }
}

// Compile (or fetch from the cache) one kernel source.
rc_status compile(const Source &s, std::vector<char> &code, std::string &key) {
    key = cache_key(s);
    std::string dir = cache_dir();
    std::string path = dir + "/" + key + ".hsaco";
    if (read_file(path, code)) return RC_OK;
    std::string src = full_source(s);
    hiprtcProgram prog;
    if (hiprtcCreateProgram(&prog, src.c_str(), (std::string(s.entry) + ".hip").c_str(), 0, nullptr,
                            nullptr) != HIPRTC_SUCCESS)
        return fail(RC_ERR_COMPILE, "hiprtcCreateProgram failed");
    std::vector<const char *> opts;
    for (auto &o : compile_options()) opts.push_back(o.c_str());
    hiprtcResult r = hiprtcCompileProgram(prog, (int)opts.size(), opts.data());
    if (r != HIPRTC_SUCCESS) {
        size_t n = 0;
        hiprtcGetProgramLogSize(prog, &n);
        std::string log(n, '\0');
        if (n) hiprtcGetProgramLog(prog, &log[0]);
        hiprtcDestroyProgram(&prog);
        return fail(RC_ERR_COMPILE, std::string("hipRTC: ") + s.entry + ": " + log.substr(0, 4000));
    }
    size_t n = 0;
    hiprtcGetCodeSize(prog, &n);
    code.resize(n);
    hiprtcGetCode(prog, code.data());
    hiprtcDestroyProgram(&prog);
    mkdirs(dir);
    std::string tmp = path + ".tmp" + std::to_string(getpid()) + "_" +
                      std::to_string(std::hash<std::thread::id>()(std::this_thread::get_id()));
    {
        std::ofstream f(tmp, std::ios::binary);
        f.write(code.data(), (std::streamsize)code.size());
    }
    rename(tmp.c_str(), path.c_str());
    return RC_OK;
}

// ---------------------------------------------------------------------
// Code-object metadata: the AMDGPU note (type 32) of the ELF holds a
// msgpack document whose "amdhsa.kernels" array has one map per kernel.
// KernelMeta reads the integer keys of the map whose ".name" is the entry.
// ---------------------------------------------------------------------
struct MsgReader {
    const unsigned char *p, *end;
    bool ok = true;
    uint64_t be(int n) {
        if (end - p < n) { ok = false; p = end; return 0; }
        uint64_t v = 0;
        for (int i = 0; i < n; ++i) v = (v << 8) | p[i];
        p += n;
        return v;
    }
    // Reads one value; strings go to *str, integers to *num (when non-null).
    // Returns the msgpack family: 'i' integer, 's' string, 'm' map (count in
    // *num, entries follow), 'a' array (count in *num), 'o' anything else
    // (consumed).
    char next(int64_t *num, std::string *str) {
        if (p >= end) { ok = false; return 'o'; }
        unsigned t = *p++;
        auto sized_str = [&](uint64_t n) {
            if ((uint64_t)(end - p) < n) { ok = false; p = end; return 'o'; }
            if (str) str->assign((const char *)p, (size_t)n);
            p += n;
            return 's';
        };
        if (t <= 0x7f) { if (num) *num = t; return 'i'; }
        if (t >= 0xe0) { if (num) *num = (int8_t)t; return 'i'; }
        if ((t & 0xf0) == 0x80) { if (num) *num = t & 0x0f; return 'm'; }
        if ((t & 0xf0) == 0x90) { if (num) *num = t & 0x0f; return 'a'; }
        if ((t & 0xe0) == 0xa0) return sized_str(t & 0x1f);
        switch (t) {
            case 0xc0: case 0xc2: case 0xc3: return 'o';
            case 0xc4: p += be(1); return 'o';
            case 0xc5: p += be(2); return 'o';
            case 0xc6: p += be(4); return 'o';
            case 0xca: p += 4; return 'o';
            case 0xcb: p += 8; return 'o';
            case 0xcc: { int64_t v = (int64_t)be(1); if (num) *num = v; return 'i'; }
            case 0xcd: { int64_t v = (int64_t)be(2); if (num) *num = v; return 'i'; }
            case 0xce: { int64_t v = (int64_t)be(4); if (num) *num = v; return 'i'; }
            case 0xcf: { int64_t v = (int64_t)be(8); if (num) *num = v; return 'i'; }
            case 0xd0: { int64_t v = (int8_t)be(1); if (num) *num = v; return 'i'; }
            case 0xd1: { int64_t v = (int16_t)be(2); if (num) *num = v; return 'i'; }
            case 0xd2: { int64_t v = (int32_t)be(4); if (num) *num = v; return 'i'; }
            case 0xd3: { int64_t v = (int64_t)be(8); if (num) *num = v; return 'i'; }
            case 0xd9: return sized_str(be(1));
            case 0xda: return sized_str(be(2));
            case 0xdb: return sized_str(be(4));
            case 0xdc: { int64_t v = (int64_t)be(2); if (num) *num = v; return 'a'; }
            case 0xdd: { int64_t v = (int64_t)be(4); if (num) *num = v; return 'a'; }
            case 0xde: { int64_t v = (int64_t)be(2); if (num) *num = v; return 'm'; }
            case 0xdf: { int64_t v = (int64_t)be(4); if (num) *num = v; return 'm'; }
        }
        ok = false;   // ext types do not occur in the metadata
        return 'o';
    }
    void skip() {
        int64_t n = 0;
        char k = next(&n, nullptr);
        if (k == 'm') n *= 2;
        if (k == 'm' || k == 'a')
            for (int64_t i = 0; i < n && ok; ++i) skip();
    }
};

struct KernelMeta {
    std::map<std::string, int64_t> ints;
    long get(const char *key) const {
        auto it = ints.find(key);
        return it == ints.end() ? -1 : (long)it->second;
    }
};

// Locate the metadata note of a 64-bit little-endian ELF code object.
bool metadata_note(const std::vector<char> &code, const unsigned char **b, const unsigned char **e) {
    const unsigned char *c = (const unsigned char *)code.data();
    const size_t n = code.size();
    if (n < 64 || memcmp(c, "\x7f" "ELF", 4) != 0 || c[4] != 2) return false;
    auto rd = [&](size_t off, int bytes) -> uint64_t {
        uint64_t v = 0;
        if (off + bytes > n) return 0;
        for (int i = bytes - 1; i >= 0; --i) v = (v << 8) | c[off + i];
        return v;
    };
    const uint64_t shoff = rd(0x28, 8), shentsize = rd(0x3a, 2), shnum = rd(0x3c, 2);
    for (uint64_t i = 0; i < shnum; ++i) {
        const size_t sh = (size_t)(shoff + i * shentsize);
        if (rd(sh + 4, 4) != 7) continue;   // SHT_NOTE
        size_t off = (size_t)rd(sh + 0x18, 8), end = off + (size_t)rd(sh + 0x20, 8);
        if (end > n) continue;
        while (off + 12 <= end) {
            const uint64_t namesz = rd(off, 4), descsz = rd(off + 4, 4), type = rd(off + 8, 4);
            const size_t name = off + 12, desc = name + ((namesz + 3) & ~3ull);
            if (desc + descsz > end) break;
            if (type == 32 && namesz >= 6 && memcmp(c + name, "AMDGPU", 6) == 0) {
                *b = c + desc;
                *e = c + desc + descsz;
                return true;
            }
            off = desc + ((descsz + 3) & ~3ull);
        }
    }
    return false;
}

// Integer keys of the metadata map of kernel `entry` (empty if not found).
KernelMeta kernel_meta(const std::vector<char> &code, const char *entry) {
    KernelMeta out;
    const unsigned char *b = nullptr, *e = nullptr;
    if (!metadata_note(code, &b, &e)) return out;
    MsgReader r{b, e};
    int64_t n = 0;
    if (r.next(&n, nullptr) != 'm') return out;
    for (int64_t i = 0; i < n && r.ok; ++i) {
        std::string key;
        if (r.next(nullptr, &key) != 's') return out;
        if (key != "amdhsa.kernels") {
            r.skip();
            continue;
        }
        int64_t nk = 0;
        if (r.next(&nk, nullptr) != 'a') return out;
        for (int64_t k = 0; k < nk && r.ok; ++k) {
            int64_t nf = 0;
            if (r.next(&nf, nullptr) != 'm') return out;
            KernelMeta m;
            std::string name;
            for (int64_t f = 0; f < nf && r.ok; ++f) {
                std::string fk;
                if (r.next(nullptr, &fk) != 's') return out;
                int64_t v = 0;
                std::string sv;
                const unsigned char *at = r.p;
                char kind = r.next(&v, &sv);
                if (kind == 'i') {
                    m.ints[fk] = v;
                } else if (kind == 's') {
                    if (fk == ".name") name = sv;
                } else if (kind == 'm' || kind == 'a') {
                    r.p = at;
                    r.skip();
                }
            }
            if (name == entry) return m;
        }
        return out;
    }
    return out;
}

// A kernel that needs private (scratch) memory spills registers: the
// schedule is illegal.  Missing metadata is a compile error.
rc_status check_spill(const std::vector<char> &code, const char *entry) {
    const KernelMeta m = kernel_meta(code, entry);
    const long scratch = m.get(".private_segment_fixed_size");
    if (scratch < 0) return fail(RC_ERR_COMPILE, std::string("no metadata for kernel ") + entry);
    if (scratch > 0)
        return fail(RC_ERR_ILLEGAL_SCHEDULE, std::string("spill: ") + entry + " needs " +
                                                 std::to_string(scratch) + " B of scratch memory per lane");
    return RC_OK;
}

std::string def(const char *name, long long v) {
    return std::string("#define ") + name + " " + std::to_string(v) + "\n";
}

// ---------------------------------------------------------------------
// Plan description: the kernels of one operator execution.
// ---------------------------------------------------------------------
struct Kern {
    Source src;
    dim3 grid, block;
    double flops = 0;   // algorithmic FLOPs of this launch (contractions only)
    // fills the argument block from the caller's buffers and the workspace
    std::function<void(const rc_args *, char *ws, ArgBlob &blob)> bind;
    hipFunction_t fn = nullptr;
};

struct WsLayout {
    size_t total = 0;
    std::map<std::string, std::pair<size_t, size_t>> parts;
    size_t add(size_t bytes, const char *name) {
        size_t off = total;
        total += (bytes + 255) & ~(size_t)255;
        parts[name] = {off, bytes};
        return off;
    }
};

struct GemmCfg {
    int tm, tn, tk, wm, wn, mf, st, vec, un, lay, grid, occ;
    int skip;   // MoE only: partial tiles skip their empty row blocks
};

GemmCfg read_block(const rc_op_desc *d, const rc_schedule *s, const char *prefix) {
    auto k = [&](const char *n) { return kv(d, s, (std::string(prefix) + n).c_str()); };
    return GemmCfg{k("tile_m"), k("tile_n"), k("tile_k"), k("waves_m"), k("waves_n"), k("mfma"),
                   k("stages"), k("vec"), k("unroll"), k("layout"), k("grid"), k("occ"),
                   std::max(0, k("skip"))};
}

std::string gemm_defs(const GemmCfg &g, int nb, int amode, int epi, long gm, long gn, long gk) {
    std::string s;
    s += def("TM", g.tm) + def("TN", g.tn) + def("TK", g.tk) + def("WM", g.wm) + def("WN", g.wn);
    s += def("MF", g.mf) + def("STAGES", g.st) + def("VEC", g.vec) + def("UNROLL", g.un);
    s += def("LAYOUT", g.lay) + def("GRID", g.grid) + def("NB", nb) + def("AMODE", amode);
    s += def("EPI", epi) + def("GM", gm) + def("GN", gn) + def("GK", gk) + def("OCC", g.occ);
    if (g.skip) s += def("ROWSKIP", 1);
    if (g.st == 7) s += def("NSTAGE", gemm_ring_stages(g.tm, g.tn, g.tk, nb, g.wm * g.wn, g.occ));
    return s;
}

template <class T>
void put(ArgBlob &blob, const T &v) {
    static_assert(sizeof(T) <= sizeof(blob.data), "kernel argument block too large");
    blob.size = sizeof(T);
    memcpy(blob.data, &v, sizeof(T));
}

}  // namespace

struct rc_plan {
    rc_op_desc desc;
    rc_schedule sched;
    std::vector<Kern> kerns;
    size_t workspace = 0;
    int dominant = 0;
    // named parts of the workspace: name -> (byte offset, bytes)
    std::map<std::string, std::pair<size_t, size_t>> parts;
};

namespace rc {

std::string cache_dir() {
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_cache_dir.empty()) return g_cache_dir;
    const char *e = getenv("RC_CACHE_DIR");
    if (e && *e) return e;
    return lib_dir() + "/jit_cache";
}

}  // namespace rc

namespace {

// Build the kernel list of a plan (no compilation, no GPU).
rc_status describe(const rc_op_desc *d, const rc_schedule *s, rc_plan &p) {
    const int64_t *D = d->dim;
    WsLayout ws;
    switch (d->kind) {
        case RC_OP_GEMM_F32: {
            int tm = kv(d, s, "tile_m"), tn = kv(d, s, "tile_n");
            int nt = 64 * kv(d, s, "waves_m") * kv(d, s, "waves_n");
            int st = kv(d, s, "stages"), sp = kv(d, s, "splits");
            Kern k;
            k.src = Source{SRC_gemm_f32, "rc_gemm_f32", ""};
            k.src.defines = def("TM", tm) + def("TN", tn) + def("TK", kv(d, s, "tile_k")) +
                            def("WM", kv(d, s, "waves_m")) + def("WN", kv(d, s, "waves_n")) +
                            def("VEC", kv(d, s, "vec")) + def("STAGES", st) +
                            def("UNROLL", kv(d, s, "unroll")) + def("LAYOUT", kv(d, s, "layout")) +
                            def("SPLITS", sp) + def("GM", D[0]) + def("GN", D[1]) + def("GK", D[2]);
            // streaming stage: one workgroup per (64-column tile, K split);
            // with K splits the per-split partial sums live in the workspace
            const bool split = st == 3 && sp > 1;
            size_t offP = split ? ws.add((size_t)sp * D[0] * D[1] * 4, "splitk.partials") : 0;
            if (st == 3)
                k.grid = dim3((unsigned)(D[1] / 64 * sp), 1, 1);
            else
                k.grid = dim3((unsigned)((D[1] + tn - 1) / tn), (unsigned)((D[0] + tm - 1) / tm), 1);
            k.block = dim3(nt, 1, 1);
            k.flops = 2.0 * D[0] * D[1] * D[2];
            k.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, GemmF32Args{a->in[0], a->in[1], a->out[0], split ? w + offP : nullptr});
            };
            p.kerns.push_back(k);
            p.dominant = 0;
            if (split) {
                Kern kr = k;
                kr.flops = 0;
                kr.src.entry = "rc_gemm_f32_splitk_reduce";
                kr.grid = dim3((unsigned)((D[0] * D[1] / 4 + 63) / 64), 1, 1);
                kr.block = dim3(256, 1, 1);
                p.kerns.push_back(kr);
            }
            break;
        }
        case RC_OP_GATED_MLP: {
            long T = D[0], Hd = D[1], I = D[2];
            GemmCfg up = read_block(d, s, "up."), dn = read_block(d, s, "down.");
            int fuse = kv(d, s, "fuse");
            // column split of a block over a main and a tail launch
            int64_t up_main = I / up.tn, up_tail = 0, dn_main = Hd / dn.tn, dn_tail = 0;
            const int up_tmode = kv(d, s, "up.tail"), dn_tmode = kv(d, s, "down.tail");
            if (up_tmode >= 1)
                gemm_tail_split(up.tm, up.tn, up.tk, 2, up.wm * up.wn, up.occ, up.st, T, I, &up_main, &up_tail);
            if (dn_tmode >= 1)
                gemm_tail_split(dn.tm, dn.tn, dn.tk, 1, dn.wm * dn.wn, dn.occ, dn.st, T, Hd, &dn_main, &dn_tail);
            auto cols = [](int64_t first, int64_t count) {
                return def("NT_FIRST", first) + def("NT_COUNT", count);
            };
            size_t offH = ws.add((size_t)T * I * 2, "hidden");
            size_t offG = 0, offU = 0;
            if (!fuse) {
                offG = ws.add((size_t)T * I * 4, "gate.f32");
                offU = ws.add((size_t)T * I * 4, "up.f32");
            }
            Kern k1;
            k1.src = Source{SRC_gemm_bf16, "rc_gemm_bf16",
                            gemm_defs(up, 2, 0, fuse ? 2 : 3, T, I, Hd) + cols(0, up_main)};
            k1.grid = dim3((unsigned)(((T + up.tm - 1) / up.tm) * up_main), 1, 1);
            k1.block = dim3(64 * up.wm * up.wn, 1, 1);
            k1.flops = 4.0 * T * Hd * up_main * up.tn;
            k1.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                if (fuse)
                    put(b, GemmBf16Args{a->in[0], a->in[1], a->in[2], w + offH, nullptr, nullptr,
                                        nullptr, nullptr, nullptr});
                else
                    put(b, GemmBf16Args{a->in[0], a->in[1], a->in[2], w + offG, w + offU, nullptr,
                                        nullptr, nullptr, nullptr});
            };
            p.kerns.push_back(k1);
            if (up_tail > 0 && up_tmode == 1) {
                GemmCfg h = up;
                h.tm /= 2;
                Kern kt = k1;
                kt.src.defines = gemm_defs(h, 2, 0, fuse ? 2 : 3, T, I, Hd) + cols(up_main, up_tail);
                kt.grid = dim3((unsigned)(((T + h.tm - 1) / h.tm) * up_tail), 1, 1);
                kt.flops = 4.0 * T * Hd * up_tail * up.tn;
                p.kerns.push_back(kt);
            }
            if (up_tail > 0 && up_tmode == 2) {
                // full tiles, K range cut in two: fp32 gate and up partial
                // sums of the tail columns, then SiLU(g) * u into the hidden
                const long wc = up_tail * up.tn;
                size_t offTG = ws.add((size_t)2 * T * wc * 4, "up.tail.gate"),
                       offTU = ws.add((size_t)2 * T * wc * 4, "up.tail.up");
                Kern kt = k1;
                kt.src.defines = gemm_defs(up, 2, 0, 3, T, I, Hd) + cols(up_main, up_tail) + def("SPLITK", 2);
                kt.grid = dim3((unsigned)(((T + up.tm - 1) / up.tm) * up_tail * 2), 1, 1);
                kt.flops = 4.0 * T * Hd * up_tail * up.tn;
                kt.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                    put(b, GemmBf16Args{a->in[0], a->in[1], a->in[2], w + offTG, w + offTU, nullptr,
                                        nullptr, nullptr, nullptr});
                };
                p.kerns.push_back(kt);
                Kern ks;
                ks.src = Source{SRC_aux, "rc_splitk_swiglu_bf16",
                                def("EW_N", T * wc) + def("EW_COLS", wc) + def("EW_LD", I) +
                                    def("EW_C0", up_main * up.tn) + def("EW_SPLITS", 2)};
                ks.grid = dim3((unsigned)((T * wc / 8 + 255) / 256), 1, 1);
                ks.block = dim3(256, 1, 1);
                ks.bind = [=](const rc_args *, char *w, ArgBlob &b) {
                    put(b, EwArgs{w + offTG, w + offTU, nullptr, w + offH});
                };
                p.kerns.push_back(ks);
            }
            if (!fuse) {
                Kern ke;
                ke.src = Source{SRC_aux, "rc_swiglu_f32", def("EW_N", T * I) + def("EW_COLS", I)};
                ke.grid = dim3((unsigned)((T * I / 4 + 255) / 256), 1, 1);
                ke.block = dim3(256, 1, 1);
                ke.bind = [=](const rc_args *, char *w, ArgBlob &b) {
                    put(b, EwArgs{w + offG, w + offU, nullptr, w + offH});
                };
                p.kerns.push_back(ke);
            }
            // K split of the down projection: SPLITK copies of the tile grid
            // store fp32 partial sums, a separate kernel adds them
            const int sk = std::max(1, kv(d, s, "down.split"));
            size_t offP = sk > 1 ? ws.add((size_t)sk * T * Hd * 4, "down.partials") : 0;
            Kern k2;
            k2.src = Source{SRC_gemm_bf16, "rc_gemm_bf16",
                            gemm_defs(dn, 1, 0, sk > 1 ? 3 : 0, T, Hd, I) + cols(0, dn_main) +
                                (sk > 1 ? def("SPLITK", sk) : std::string())};
            k2.grid = dim3((unsigned)(((T + dn.tm - 1) / dn.tm) * dn_main * sk), 1, 1);
            k2.block = dim3(64 * dn.wm * dn.wn, 1, 1);
            k2.flops = 2.0 * T * I * dn_main * dn.tn;
            k2.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, GemmBf16Args{w + offH, a->in[3], nullptr, sk > 1 ? w + offP : a->out[0], nullptr,
                                    nullptr, nullptr, nullptr, nullptr});
            };
            p.kerns.push_back(k2);
            if (sk > 1) {
                Kern kr;
                kr.src = Source{SRC_aux, "rc_splitk_sum_bf16",
                                def("EW_N", T * Hd) + def("EW_COLS", Hd) + def("EW_SPLITS", sk)};
                kr.grid = dim3((unsigned)((T * Hd / 8 + 255) / 256), 1, 1);
                kr.block = dim3(256, 1, 1);
                kr.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                    put(b, EwArgs{w + offP, nullptr, nullptr, a->out[0]});
                };
                p.kerns.push_back(kr);
            }
            if (dn_tail > 0 && dn_tmode == 1) {
                GemmCfg h = dn;
                h.tm /= 2;
                Kern kt = k2;
                kt.src.defines = gemm_defs(h, 1, 0, 0, T, Hd, I) + cols(dn_main, dn_tail);
                kt.grid = dim3((unsigned)(((T + h.tm - 1) / h.tm) * dn_tail), 1, 1);
                kt.flops = 2.0 * T * I * dn_tail * dn.tn;
                p.kerns.push_back(kt);
            }
            if (dn_tail > 0 && dn_tmode == 2) {
                const long wc = dn_tail * dn.tn;
                size_t offTP = ws.add((size_t)2 * T * wc * 4, "down.tail.partials");
                Kern kt = k2;
                kt.src.defines = gemm_defs(dn, 1, 0, 3, T, Hd, I) + cols(dn_main, dn_tail) + def("SPLITK", 2);
                kt.grid = dim3((unsigned)(((T + dn.tm - 1) / dn.tm) * dn_tail * 2), 1, 1);
                kt.flops = 2.0 * T * I * dn_tail * dn.tn;
                kt.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                    put(b, GemmBf16Args{w + offH, a->in[3], nullptr, w + offTP, nullptr, nullptr,
                                        nullptr, nullptr, nullptr});
                };
                p.kerns.push_back(kt);
                Kern ks;
                ks.src = Source{SRC_aux, "rc_splitk_sum_bf16",
                                def("EW_N", T * wc) + def("EW_COLS", wc) + def("EW_LD", Hd) +
                                    def("EW_C0", dn_main * dn.tn) + def("EW_SPLITS", 2)};
                ks.grid = dim3((unsigned)((T * wc / 8 + 255) / 256), 1, 1);
                ks.block = dim3(256, 1, 1);
                ks.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                    put(b, EwArgs{w + offTP, nullptr, nullptr, a->out[0]});
                };
                p.kerns.push_back(ks);
            }
            p.dominant = 0;
            break;
        }
        case RC_OP_MOE: {
            long T = D[0], Hd = D[1], E = D[2], I = D[3], topk = D[4], R = T * topk;
            GemmCfg up = read_block(d, s, "up."), dn = read_block(d, s, "down.");
            int fuse = kv(d, s, "fuse");
            size_t offOff = ws.add((E + 1) * 4, "offsets"), offPerm = ws.add(R * 4, "perm");
            size_t offPos = ws.add(R * 4, "pos");
            size_t offTu = ws.add((E + 1) * 4, "tile_up"), offTd = ws.add((E + 1) * 4, "tile_down");
            size_t offH = ws.add((size_t)R * I * 2, "hidden"), offY = ws.add((size_t)R * Hd * 2, "expert_out");
            const long nblk = (R + 1023) / 1024;    // routing blocks of 1024 rows
            size_t offCnt = ws.add((size_t)nblk * E * 4, "block_counts");
            size_t offG = 0, offU = 0;
            if (!fuse) {
                offG = ws.add((size_t)R * I * 4, "gate.f32");
                offU = ws.add((size_t)R * I * 4, "up.f32");
            }
            std::string moe = def("MOE_T", T) + def("MOE_TOPK", topk) + def("MOE_E", E) +
                              def("MOE_H", Hd) + def("MOE_TM_UP", up.tm) + def("MOE_TM_DOWN", dn.tm);
            // routing: per-block expert histograms, then the stable scatter
            Kern kh;
            kh.src = Source{SRC_aux, "rc_moe_hist", moe};
            kh.grid = dim3((unsigned)nblk, 1, 1);
            kh.block = dim3(1024, 1, 1);
            kh.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, MoeHistArgs{a->in[1], w + offCnt});
            };
            p.kerns.push_back(kh);
            Kern k0;
            k0.src = Source{SRC_aux, "rc_moe_prep", moe};
            k0.grid = dim3((unsigned)nblk, 1, 1);
            k0.block = dim3(1024, 1, 1);
            k0.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, MoePrepArgs{a->in[1], w + offCnt, w + offOff, w + offPerm, w + offPos, w + offTu,
                                   w + offTd});
            };
            p.kerns.push_back(k0);
            std::string mdefs = def("TOPK", topk) + def("NEXP", E);
            Kern k1;
            k1.src = Source{SRC_gemm_bf16, "rc_gemm_bf16",
                            gemm_defs(up, 2, 1, fuse ? 2 : 3, R, I, Hd) + mdefs};
            long ntm_up = (R + up.tm - 1) / up.tm + E;
            k1.grid = dim3((unsigned)(ntm_up * (I / up.tn)), 1, 1);
            k1.block = dim3(64 * up.wm * up.wn, 1, 1);
            k1.flops = 4.0 * R * Hd * I;
            k1.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, GemmBf16Args{a->in[0], a->in[3], a->in[4], w + (fuse ? offH : offG),
                                    fuse ? nullptr : w + offU, nullptr, w + offPerm, w + offOff,
                                    w + offTu});
            };
            p.kerns.push_back(k1);
            p.dominant = 2;
            if (!fuse) {
                Kern ke;
                ke.src = Source{SRC_aux, "rc_swiglu_f32", def("EW_N", R * I) + def("EW_COLS", I)};
                ke.grid = dim3((unsigned)((R * I / 4 + 255) / 256), 1, 1);
                ke.block = dim3(256, 1, 1);
                ke.bind = [=](const rc_args *, char *w, ArgBlob &b) {
                    put(b, EwArgs{w + offG, w + offU, nullptr, w + offH});
                };
                p.kerns.push_back(ke);
            }
            Kern k2;
            k2.src = Source{SRC_gemm_bf16, "rc_gemm_bf16", gemm_defs(dn, 1, 3, 0, R, Hd, I) + mdefs};
            long ntm_dn = (R + dn.tm - 1) / dn.tm + E;
            k2.grid = dim3((unsigned)(ntm_dn * (Hd / dn.tn)), 1, 1);
            k2.block = dim3(64 * dn.wm * dn.wn, 1, 1);
            k2.flops = 2.0 * R * I * Hd;
            k2.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, GemmBf16Args{w + offH, a->in[5], nullptr, w + offY, nullptr, nullptr,
                                    w + offPerm, w + offOff, w + offTd});
            };
            p.kerns.push_back(k2);
            Kern k3;
            k3.src = Source{SRC_aux, "rc_moe_combine", moe};
            k3.grid = dim3((unsigned)((T * (Hd / 8) + 255) / 256), 1, 1);
            k3.block = dim3(256, 1, 1);
            k3.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                put(b, MoeCombineArgs{w + offY, w + offPos, a->in[2], a->out[0]});
            };
            p.kerns.push_back(k3);
            break;
        }
        case RC_OP_CONV2D: {
            long N = D[0], H = D[1], W = D[2], C = D[3], K = D[4], R = D[5], S = D[6], pad = D[7];
            long P = H + 2 * pad - R + 1, Q = W + 2 * pad - S + 1, M = N * P * Q;
            GemmCfg g = read_block(d, s, "");
            int fuse = kv(d, s, "fuse");
            const bool act = (d->flags & RC_FLAG_NO_ACT) == 0;
            size_t offPre = fuse ? 0 : ws.add((size_t)M * K * 4, "pre.f32");
            std::string cv = def("CV_H", H) + def("CV_W", W) + def("CV_C", C) + def("CV_P", P) +
                             def("CV_Q", Q) + def("CV_S", S) + def("CV_PAD", pad);
            Kern k1;
            k1.src = Source{SRC_gemm_bf16, "rc_gemm_bf16",
                            gemm_defs(g, 1, 2, fuse ? (act ? 1 : 4) : 3, M, K, R * S * C) + cv};
            k1.grid = dim3((unsigned)(((M + g.tm - 1) / g.tm) * (K / g.tn)), 1, 1);
            k1.block = dim3(64 * g.wm * g.wn, 1, 1);
            k1.flops = 2.0 * M * K * R * S * C;
            k1.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                if (fuse)
                    put(b, GemmBf16Args{a->in[0], a->in[1], nullptr, a->out[0], nullptr, a->in[2],
                                        nullptr, nullptr, nullptr});
                else
                    put(b, GemmBf16Args{a->in[0], a->in[1], nullptr, w + offPre, nullptr, nullptr,
                                        nullptr, nullptr, nullptr});
            };
            p.kerns.push_back(k1);
            if (!fuse) {
                Kern ke;
                ke.src = Source{SRC_aux, "rc_bias_silu_f32",
                                def("EW_N", M * K) + def("EW_COLS", K) + def("EW_ACT", act ? 1 : 0)};
                ke.grid = dim3((unsigned)((M * K / 4 + 255) / 256), 1, 1);
                ke.block = dim3(256, 1, 1);
                ke.bind = [=](const rc_args *a, char *w, ArgBlob &b) {
                    put(b, EwArgs{w + offPre, nullptr, a->in[2], a->out[0]});
                };
                p.kerns.push_back(ke);
            }
            p.dominant = 0;
            break;
        }
        case RC_OP_ATTENTION: {
            long B = D[0], Hh = D[1], S = D[2], Dh = D[3];
            int bm = kv(d, s, "block_m"), bn = kv(d, s, "block_n"), w = kv(d, s, "waves");
            int mf = kv(d, s, "mfma"), chunk = kv(d, s, "chunk");
            bool causal = (d->flags & RC_FLAG_CAUSAL) != 0;
            // work items: query tile t sees tiles(t) key tiles, cut into
            // chunks of at most `chunk` tiles
            // (the last query and key tiles may be partial)
            long nqt = (S + bm - 1) / bm, nkt = (S + bn - 1) / bn, items = 0, maxch = 1;
            for (long t = 0; t < nqt; ++t) {
                long tiles = causal ? std::min(nkt, (t * bm + bm - 1) / bn + 1) : nkt;
                long nc = chunk > 0 ? (tiles + chunk - 1) / chunk : 1;
                items += nc;
                maxch = std::max(maxch, nc);
            }
            // partial state per (head, query tile, chunk): for every wave, m
            // and l of its rows, then its output accumulators
            long qb = bm / w / mf, accn = mf == 16 ? 4 : 16;
            long wslot = qb * 2 * mf + qb * (Dh / mf) * accn * 64;
            size_t offP = chunk > 0 ? ws.add((size_t)B * Hh * nqt * maxch * w * wslot * 4, "partials") : 0;
            Kern k;
            double scale_log2 = 1.4426950408889634 / std::sqrt((double)Dh);
            char sbuf[64];
            snprintf(sbuf, sizeof sbuf, "#define SCALE_LOG2 %.17gf\n", scale_log2);
            k.src = Source{SRC_attention, "rc_attention",
                           def("BM", bm) + def("BN", bn) + def("NW", w) +
                               def("MF", mf) + def("STAGES", kv(d, s, "stages")) +
                               def("VEC", kv(d, s, "vec")) + def("UNROLL", kv(d, s, "unroll")) +
                               def("ORDER", kv(d, s, "order")) + def("OCC", kv(d, s, "occ")) +
                               def("SPLITS", kv(d, s, "splits")) + def("CHUNK", chunk) +
                               def("AB", B) + def("AH", Hh) +
                               def("AS", S) + def("AD", Dh) +
                               def("CAUSAL", causal ? 1 : 0) + sbuf};
            k.grid = dim3((unsigned)(B * Hh * items), 1, 1);
            k.block = dim3(64 * w * kv(d, s, "splits"), 1, 1);
            k.flops = rc_op_flops(d);
            k.bind = [=](const rc_args *a, char *ws_base, ArgBlob &b) {
                put(b, AttnArgs{a->in[0], a->in[1], a->in[2], a->out[0], chunk > 0 ? ws_base + offP : nullptr});
            };
            p.kerns.push_back(k);
            if (chunk > 0) {
                Kern kc = k;
                kc.flops = 0;
                kc.src.entry = "rc_attention_combine";
                kc.grid = dim3((unsigned)(B * Hh * nqt), 1, 1);
                kc.block = dim3(64 * w, 1, 1);
                p.kerns.push_back(kc);
            }
            p.dominant = 0;
            break;
        }
        default: return fail(RC_ERR_UNSUPPORTED, "unknown operator kind");
    }
    p.workspace = ws.total;
    p.parts = ws.parts;
    return RC_OK;
}

int n_inputs(int kind) {
    switch (kind) {
        case RC_OP_GEMM_F32: return 2;
        case RC_OP_ATTENTION: return 3;
        case RC_OP_GATED_MLP: return 4;
        case RC_OP_MOE: return 6;
        case RC_OP_CONV2D: return 3;
    }
    return 0;
}

rc_status hip_fail(hipError_t e, const char *what) {
    return fail(RC_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Cache-flush buffers of rc_time, one per device (allocated on the first
// flushed timing on that device, freed by rc_time_release).
std::map<int, void *> g_flush;
const size_t FLUSH_BYTES = (size_t)512 << 20;

rc_status flush_buffer(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    std::lock_guard<std::mutex> g(g_mu);
    auto it = g_flush.find(dev);
    if (it != g_flush.end()) {
        *out = it->second;
        return RC_OK;
    }
    void *p = nullptr;
    e = hipMalloc(&p, FLUSH_BYTES);
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(flush buffer)");
    g_flush[dev] = p;
    *out = p;
    return RC_OK;
}

}  // namespace

extern "C" {

rc_status rc_set_cache_dir(const char *dir) {
    std::lock_guard<std::mutex> g(g_mu);
    g_cache_dir = dir ? dir : "";
    return RC_OK;
}

rc_status rc_precompile(const rc_op_desc *d, const rc_schedule *s, int32_t n, int32_t nthreads,
                        rc_status *status) {
    if (!desc_ok(d) || (!s && n > 0) || n < 0) return fail(RC_ERR_INVALID_ARGUMENT, "bad arguments");
    std::atomic<int> next(0);
    std::atomic<int> nfail(0);
    std::vector<rc_status> st(n, RC_OK);
    auto work = [&]() {
        for (;;) {
            int i = next.fetch_add(1);
            if (i >= n) return;
            std::string why = check_schedule(d, &s[i]);
            if (!why.empty()) {
                st[i] = RC_ERR_ILLEGAL_SCHEDULE;
                ++nfail;
                continue;
            }
            rc_plan p;
            rc_status r = describe(d, &s[i], p);
            for (auto &k : p.kerns) {
                if (r != RC_OK) break;
                std::vector<char> code;
                std::string key;
                r = compile(k.src, code, key);
                if (r == RC_OK) r = check_spill(code, k.src.entry);
            }
            st[i] = r;
            if (r != RC_OK) ++nfail;
        }
    };
    int nt = std::max(1, std::min<int>(nthreads, n));
    std::vector<std::thread> pool;
    for (int t = 0; t < nt; ++t) pool.emplace_back(work);
    for (auto &t : pool) t.join();
    if (status)
        for (int i = 0; i < n; ++i) status[i] = st[i];
    if (nfail) return fail(RC_ERR_COMPILE, std::to_string(nfail.load()) + " of " + std::to_string(n) +
                                               " schedules failed to compile or are illegal");
    return RC_OK;
}

rc_status rc_describe(const rc_op_desc *d, const rc_schedule *s, rc_kernel_info *buf, int32_t cap,
                      int32_t *n) {
    if (!desc_ok(d) || !s || !n) return fail(RC_ERR_INVALID_ARGUMENT, "bad arguments");
    std::string why = check_schedule(d, s);
    if (!why.empty()) return fail(RC_ERR_ILLEGAL_SCHEDULE, why);
    rc_plan p;
    rc_status r = describe(d, s, p);
    if (r != RC_OK) return r;
    *n = (int32_t)p.kerns.size();
    for (int32_t i = 0; i < *n; ++i) {
        std::vector<char> code;
        std::string key;
        r = compile(p.kerns[i].src, code, key);
        if (r != RC_OK) return r;
        if (!buf || i >= cap) continue;
        rc_kernel_info k;
        memset(&k, 0, sizeof k);
        k.struct_size = sizeof k;
        snprintf(k.name, sizeof k.name, "%s", p.kerns[i].src.entry);
        const Kern &kk = p.kerns[i];
        k.grid = (int32_t)(kk.grid.x * kk.grid.y * kk.grid.z);
        k.block = (int32_t)(kk.block.x * kk.block.y * kk.block.z);
        const KernelMeta m = kernel_meta(code, p.kerns[i].src.entry);
        if (m.ints.empty())
            return fail(RC_ERR_COMPILE, std::string("no metadata for kernel ") + p.kerns[i].src.entry);
        k.lds_bytes = (int32_t)m.get(".group_segment_fixed_size");
        k.vgprs = (int32_t)m.get(".vgpr_count");
        k.agprs = (int32_t)m.get(".agpr_count");
        k.sgprs = (int32_t)m.get(".sgpr_count");
        k.scratch_bytes = (int32_t)m.get(".private_segment_fixed_size");
        // Occupancy on gfx950: 512 registers per lane per SIMD shared by the
        // resident waves (the metadata's vgpr_count is the combined VGPR +
        // AGPR allocation), allocated in blocks of 8, at most 8 waves per
        // SIMD; LDS of 160 KiB per CU shared by the resident workgroups.
        int regs = std::max(k.vgprs, 0);
        regs = (regs + 7) / 8 * 8;
        int by_regs = regs > 0 ? std::min(8, 512 / regs) : 8;
        int waves_per_wg = (k.block + 63) / 64;
        int wg_per_cu = k.lds_bytes > 0 ? 163840 / k.lds_bytes : 32;
        int by_lds = std::max(1, wg_per_cu * waves_per_wg / 4);   // 4 SIMDs per CU
        k.waves_per_simd = std::min(by_regs, by_lds);
        buf[i] = k;
    }
    return RC_OK;
}

rc_status rc_plan_create(const rc_op_desc *d, const rc_schedule *s, rc_plan **out) {
    if (!desc_ok(d) || !s || !out) return fail(RC_ERR_INVALID_ARGUMENT, "bad arguments");
    *out = nullptr;
    std::string why = check_schedule(d, s);
    if (!why.empty()) return fail(RC_ERR_ILLEGAL_SCHEDULE, why);
    std::unique_ptr<rc_plan> p(new rc_plan());
    p->desc = *d;
    p->sched = *s;
    rc_status r = describe(d, s, *p);
    if (r != RC_OK) return r;
    for (auto &k : p->kerns) {
        std::vector<char> code;
        std::string key;
        r = compile(k.src, code, key);
        if (r != RC_OK) return r;
        r = check_spill(code, k.src.entry);
        if (r != RC_OK) return r;
        hipModule_t mod;
        {
            std::lock_guard<std::mutex> g(g_mu);
            int dev = 0;
            if (hipGetDevice(&dev) != hipSuccess) dev = -1;
            std::string mkey = key + "@" + std::to_string(dev);
            auto it = g_modules.find(mkey);
            if (it == g_modules.end()) {
                hipError_t e = hipModuleLoadData(&mod, code.data());
                if (e != hipSuccess) return hip_fail(e, "hipModuleLoadData");
                g_modules[mkey] = mod;
            } else {
                mod = it->second;
            }
        }
        hipError_t e = hipModuleGetFunction(&k.fn, mod, k.src.entry);
        if (e != hipSuccess) return hip_fail(e, "hipModuleGetFunction");
    }
    *out = p.release();
    clear_error();
    return RC_OK;
}

void rc_plan_destroy(rc_plan *p) { delete p; }

rc_status rc_plan_workspace(const rc_plan *p, size_t *bytes) {
    if (!p || !bytes) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    *bytes = p->workspace;
    return RC_OK;
}

rc_status rc_plan_kernels(const rc_plan *p, int32_t *nkernels, int32_t *dominant) {
    if (!p) return fail(RC_ERR_INVALID_ARGUMENT, "null plan");
    if (nkernels) *nkernels = (int32_t)p->kerns.size();
    if (dominant) *dominant = p->dominant;
    return RC_OK;
}

rc_status rc_plan_kernel_flops(const rc_plan *p, int32_t kernel, double *flops) {
    if (!p || !flops) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    if (kernel < 0 || kernel >= (int32_t)p->kerns.size()) return fail(RC_ERR_INVALID_ARGUMENT, "kernel index out of range");
    *flops = p->kerns[kernel].flops;
    return RC_OK;
}

rc_status rc_plan_buffer(const rc_plan *p, const char *name, size_t *offset, size_t *bytes) {
    if (!p || !name || !offset || !bytes) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    auto it = p->parts.find(name);
    if (it == p->parts.end()) return fail(RC_ERR_INVALID_ARGUMENT, std::string("no workspace part named ") + name);
    *offset = it->second.first;
    *bytes = it->second.second;
    return RC_OK;
}

rc_status rc_time_release(void) {
    std::lock_guard<std::mutex> g(g_mu);
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    rc_status r = RC_OK;
    for (auto &kv : g_flush) {
        if ((e = hipSetDevice(kv.first)) != hipSuccess || (e = hipFree(kv.second)) != hipSuccess)
            r = hip_fail(e, "hipFree(flush buffer)");
    }
    g_flush.clear();
    (void)hipSetDevice(cur);
    return r;
}

static rc_status check_args(const rc_plan *p, const rc_args *a, void *ws, size_t ws_bytes) {
    if (!p || !a || a->struct_size < sizeof(rc_args)) return fail(RC_ERR_INVALID_ARGUMENT, "null plan or args");
    int ni = n_inputs(p->desc.kind);
    for (int i = 0; i < ni; ++i) {
        if (!a->in[i]) return fail(RC_ERR_INVALID_ARGUMENT, "input " + std::to_string(i) + " is NULL");
        if ((uintptr_t)a->in[i] & 15) return fail(RC_ERR_MISALIGNED, "input " + std::to_string(i) + " is not 16-byte aligned");
    }
    if (!a->out[0]) return fail(RC_ERR_INVALID_ARGUMENT, "output is NULL");
    if ((uintptr_t)a->out[0] & 15) return fail(RC_ERR_MISALIGNED, "output is not 16-byte aligned");
    if (p->workspace) {
        if (!ws || ws_bytes < p->workspace)
            return fail(RC_ERR_INVALID_ARGUMENT, "workspace of " + std::to_string(p->workspace) + " bytes required");
        if ((uintptr_t)ws & 255) return fail(RC_ERR_MISALIGNED, "workspace is not 256-byte aligned");
    }
    return RC_OK;
}

static rc_status launch_impl(const rc_plan *p, const rc_args *a, void *ws, size_t ws_bytes,
                             void *stream, void **events, int32_t nevents) {
    rc_status r = check_args(p, a, ws, ws_bytes);
    if (r != RC_OK) return r;
    if (events && nevents < (int32_t)p->kerns.size() + 1)
        return fail(RC_ERR_INVALID_ARGUMENT, "need nkernels + 1 events");
    hipStream_t st = (hipStream_t)stream;
    ArgBlob blob;
    for (size_t i = 0; i < p->kerns.size(); ++i) {
        const Kern &k = p->kerns[i];
        k.bind(a, (char *)ws, blob);
        size_t sz = blob.size;
        void *cfg[] = {HIP_LAUNCH_PARAM_BUFFER_POINTER, blob.data, HIP_LAUNCH_PARAM_BUFFER_SIZE, &sz,
                       HIP_LAUNCH_PARAM_END};
        if (events) {
            hipError_t e = hipEventRecord((hipEvent_t)events[i], st);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
        }
        hipError_t e = hipModuleLaunchKernel(k.fn, k.grid.x, k.grid.y, k.grid.z, k.block.x,
                                             k.block.y, k.block.z, 0, st, nullptr, cfg);
        if (e != hipSuccess) return hip_fail(e, (std::string("launch ") + k.src.entry).c_str());
    }
    if (events) {
        hipError_t e = hipEventRecord((hipEvent_t)events[p->kerns.size()], st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
    return RC_OK;
}

rc_status rc_launch(const rc_plan *p, const rc_args *a, void *workspace, size_t ws_bytes,
                    void *stream) {
    return launch_impl(p, a, workspace, ws_bytes, stream, nullptr, 0);
}

}  // extern "C"

namespace rc {
rc_status launch_plan(const rc_plan *p, const rc_args *a, void *workspace, size_t ws_bytes, void *stream) {
    return launch_impl(p, a, workspace, ws_bytes, stream, nullptr, 0);
}
}  // namespace rc

extern "C" {

rc_status rc_launch_timed(const rc_plan *p, const rc_args *a, void *workspace, size_t ws_bytes,
                          void *stream, void **events, int32_t nevents) {
    if (!events) return fail(RC_ERR_INVALID_ARGUMENT, "events is NULL");
    return launch_impl(p, a, workspace, ws_bytes, stream, events, nevents);
}

void rc_time_opts_init(rc_time_opts *o) {
    if (!o) return;
    o->struct_size = sizeof(rc_time_opts);
    o->warmup = 3;
    o->repeat = 20;
    o->flush = 1;
    o->reserved = 0;
}

static double quantile(std::vector<double> v, double q) {
    std::sort(v.begin(), v.end());
    if (v.empty()) return 0.0;
    double pos = q * (v.size() - 1);
    size_t lo = (size_t)pos;
    size_t hi = std::min(lo + 1, v.size() - 1);
    return v[lo] + (pos - lo) * (v[hi] - v[lo]);
}

rc_status rc_time(const rc_plan *p, const rc_args *a, void *ws, size_t ws_bytes, void *stream,
                  const rc_time_opts *o, rc_timing *out) {
    if (!p || !a || !out) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    rc_time_opts opt;
    rc_time_opts_init(&opt);
    if (o) opt = *o;
    if (opt.repeat < 1 || opt.warmup < 0) return fail(RC_ERR_INVALID_ARGUMENT, "repeat must be >= 1");
    hipStream_t st = (hipStream_t)stream;
    void *flush = nullptr;
    if (opt.flush) {
        rc_status r = flush_buffer(&flush);
        if (r != RC_OK) return r;
    }
    for (int i = 0; i < opt.warmup; ++i) {
        rc_status r = rc_launch(p, a, ws, ws_bytes, stream);
        if (r != RC_OK) return r;
    }
    int nk = (int)p->kerns.size();
    std::vector<hipEvent_t> ev;
    ev.reserve((size_t)opt.repeat * (nk + 1));
    rc_status r = RC_OK;
    for (size_t i = 0; i < (size_t)opt.repeat * (nk + 1) && r == RC_OK; ++i) {
        hipEvent_t e;
        hipError_t he = hipEventCreate(&e);
        if (he != hipSuccess)
            r = hip_fail(he, "hipEventCreate");
        else
            ev.push_back(e);
    }
    for (int i = 0; i < opt.repeat && r == RC_OK; ++i) {
        if (opt.flush) {
            hipError_t e = hipMemsetAsync(flush, i & 0xFF, FLUSH_BYTES, st);
            if (e != hipSuccess) r = hip_fail(e, "flush");
        }
        if (r == RC_OK) r = launch_impl(p, a, ws, ws_bytes, stream, (void **)&ev[(size_t)i * (nk + 1)], nk + 1);
    }
    // the events must have completed before they are read or destroyed
    hipError_t se = hipStreamSynchronize(st);
    if (r == RC_OK && se != hipSuccess) r = hip_fail(se, "hipStreamSynchronize");
    if (r == RC_OK) {
        std::vector<double> tot, per[8];
        for (int i = 0; i < opt.repeat; ++i) {
            hipEvent_t *e = &ev[(size_t)i * (nk + 1)];
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, e[0], e[nk]) != hipSuccess) r = fail(RC_ERR_HIP, "hipEventElapsedTime");
            tot.push_back(ms);
            for (int k = 0; k < nk && k < 8; ++k) {
                float km = 0.f;
                if (hipEventElapsedTime(&km, e[k], e[k + 1]) != hipSuccess) r = fail(RC_ERR_HIP, "hipEventElapsedTime");
                per[k].push_back(km);
            }
        }
        rc_timing t;
        memset(&t, 0, sizeof t);
        t.struct_size = sizeof t;
        t.nkernels = nk;
        t.median_ms = quantile(tot, 0.5);
        t.q1_ms = quantile(tot, 0.25);
        t.q3_ms = quantile(tot, 0.75);
        t.min_ms = *std::min_element(tot.begin(), tot.end());
        double sum = 0;
        for (double x : tot) sum += x;
        t.mean_ms = sum / tot.size();
        double sec = t.median_ms * 1e-3;
        t.tflops = rc_op_flops(&p->desc) / sec / 1e12;
        t.gbps = rc_op_bytes(&p->desc) / sec / 1e9;
        t.frac_flops = t.tflops * 1e12 / rc_peak_flops(&p->desc);
        t.frac_bytes = t.gbps * 1e9 / rc_peak_bytes_per_s();
        for (int k = 0; k < nk && k < 8; ++k) t.kernel_ms[k] = quantile(per[k], 0.5);
        *out = t;
    }
    for (auto &e : ev) (void)hipEventDestroy(e);
    return r;
}

}  // extern "C"
