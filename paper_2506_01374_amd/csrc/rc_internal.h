// Internal declarations shared by the host-side translation units of librc.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "rc.h"

namespace rc {

struct KnobDef {
    const char *name;
    const char *xform;        // transformation class
    std::vector<int32_t> values;
    int32_t def;              // value in the untransformed program P0
};

// Knob table of an operator kind (empty for an unknown kind).
const std::vector<KnobDef> &knobs_for(int32_t kind);
// Index of a knob by name, -1 if absent.
int knob_index(int32_t kind, const char *name);

rc_status fail(rc_status s, const std::string &msg);
void clear_error();

bool desc_ok(const rc_op_desc *d);
// Knob value by name (asserts the name exists for the kind).
int32_t kv(const rc_op_desc *d, const rc_schedule *s, const char *name);

// Depth of the direct-to-LDS ring of bf16 GEMM stages 7.
int gemm_ring_stages(int tm, int tn, int tk, int nb, int waves, int occ);

// Column split of a GEMM block over two launches (the "tail" knob).
bool gemm_tail_split(int tm, int tn, int tk, int nb, int waves, int occ, int st, int64_t M, int64_t N,
                     int64_t *main_cols, int64_t *tail_cols);

// Legality with a reason; "" when legal.
std::string check_schedule(const rc_op_desc *d, const rc_schedule *s);

// Directory holding the kernel sources' embedded copy and the cache.
std::string cache_dir();

// rc_launch with the workspace given by the caller of this function (no
// allocation on any path that succeeds).
rc_status launch_plan(const rc_plan *p, const rc_args *a, void *workspace, size_t ws_bytes,
                      void *stream);

}  // namespace rc
