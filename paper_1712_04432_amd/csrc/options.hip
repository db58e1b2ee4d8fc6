// Kernel-routing and split options of the library (declared in include/imbd.h).
//
// Each option starts from its IMBD_* environment variable, read once when the library
// is loaded, or from its default; afterwards only imbd_set_option changes it. Launches
// and workspace sizing read the current value through opt(); the environment is never
// read again, so a plan and the run that follows it see the same setting unless the
// caller changes it in between.

#include <atomic>
#include <stdlib.h>

#include "common.h"

namespace imbd {

namespace {

struct OptionDef {
  const char *env;
  int dflt, lo, hi;
};

// Indexed by enum imbd_option.
const OptionDef kOptions[IMBD_OPT_COUNT] = {
    {"IMBD_SKINNY_OFF", 0, 0, 1},        // forward / Delta_X at B <= 256 on the tiled template
    {"IMBD_SKINNY_SPLITS", 0, 0, 64},    // skinny kernel's K split (0: planner)
    {"IMBD_TOP_UNFUSED", 0, 0, 1},       // top layer's softmax in its own launch
    {"IMBD_WIDE_OFF", 0, 0, 1},          // forward / Delta_X at B > 256 on the tiled template
    {"IMBD_WIDE_SPLITS", 0, 0, 4096},    // wide-batch kernel's K split (0: planner)
    {"IMBD_DW_WIDE_MIN_K", 257, 1, 1 << 30},  // smallest batch whose fused update is large-tile
    {"IMBD_DW_STREAM", 1, 0, 1},         // persistent update past 256 samples streams Delta_Y
    {"IMBD_DW_GENERIC", 0, 0, 1},        // fused update on the tiled template
    {"IMBD_GEMM_CFG", -1, -1, 3},        // tiled template's tile configuration (-1: planner)
    {"IMBD_GEMM_SPLITS", 0, 0, 4096},    // tiled template's K split (0: planner)
    {"IMBD_CONV_NT", 1, 0, 3},           // conv tile: 0 tiled template, 1 planned, 2 / 3 128 / 112 positions
    {"IMBD_SKINNY_NB", 0, 0, 4},         // skinny kernel's samples per workgroup / 64 (0: planner)
    {"IMBD_DW_WIDE_DUAL", -1, -1, 1},    // large-tile fused update, two workgroups per CU (-1: planner)
    {"IMBD_LOCAL_PAIR", 1, 0, 1},        // local backward: Delta_X and Delta_W products in one launch
    {"IMBD_REDUCE_TAIL", 1, 0, 1},       // a Delta_X split reduce carried by the next update launch
};

std::atomic<int> g_opt[IMBD_OPT_COUNT];

struct OptionInit {
  OptionInit() {
    for (int i = 0; i < IMBD_OPT_COUNT; ++i) {
      const OptionDef &d = kOptions[i];
      int v = d.dflt;
      const char *e = getenv(d.env);
      if (e && *e) {
        const long x = strtol(e, nullptr, 10);
        if (x >= d.lo && x <= d.hi && !(i == IMBD_OPT_SKINNY_NB && x == 3)) v = (int)x;
      }
      g_opt[i].store(v, std::memory_order_relaxed);
    }
  }
};
// Defined after g_opt in this file, so it runs after g_opt exists, at library load.
OptionInit g_option_init;

}  // namespace

int opt(int key) { return g_opt[key].load(std::memory_order_relaxed); }

}  // namespace imbd

using namespace imbd;

extern "C" {

int imbd_set_option(int key, int value) {
  if (key < 0 || key >= IMBD_OPT_COUNT) {
    set_error("unknown option %d", key);
    return IMBD_EINVAL;
  }
  const OptionDef &d = kOptions[key];
  if (value < d.lo || value > d.hi || (key == IMBD_OPT_SKINNY_NB && value == 3)) {
    set_error("option %s: value %d outside [%d, %d]", d.env, value, d.lo, d.hi);
    return IMBD_EINVAL;
  }
  g_opt[key].store(value, std::memory_order_relaxed);
  return IMBD_OK;
}

int imbd_get_option(int key, int *value) {
  if (key < 0 || key >= IMBD_OPT_COUNT || !value) {
    set_error("unknown option %d or value is NULL", key);
    return IMBD_EINVAL;
  }
  *value = g_opt[key].load(std::memory_order_relaxed);
  return IMBD_OK;
}

const char *imbd_option_name(int key) {
  return (key >= 0 && key < IMBD_OPT_COUNT) ? kOptions[key].env : "";
}

}  // extern "C"
