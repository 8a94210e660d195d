// Tuning overrides: read from the environment once, at library load, and
// changed afterwards only through ds_set_tuning (see tuning.hpp).
#include "tuning.hpp"

#include <atomic>
#include <cstdlib>
#include <cstring>

#include "common.hpp"

namespace ds {
namespace {

const char *const kNames[kKnobs] = {"DS_FORCE_VARIANT",   "DS_JIT_WSPLIT", "DS_JIT_SLOTS", "DS_JIT_MAP",
                                    "DS_JIT_GROUP_TILES", "DS_JIT_ORDER",  "DS_JIT_TN",    "DS_JIT_PGROUPS",
                                    "DS_ROWS_BATCH", "DS_JIT_TRANSPOSE"};

struct Knobs {
    std::atomic<int> v[kKnobs];
    Knobs()
    {
        for (int i = 0; i < kKnobs; ++i) {
            const char *e = std::getenv(kNames[i]);
            v[i].store(e && *e ? std::atoi(e) : -1, std::memory_order_relaxed);
        }
    }
};

Knobs &knobs()
{
    static Knobs k;  // constructed at load by the initializer below, before any entry point runs
    return k;
}

const Knobs &g_loaded = knobs();

int find(const char *name)
{
    for (int i = 0; i < kKnobs; ++i)
        if (std::strcmp(name, kNames[i]) == 0) return i;
    return -1;
}

}  // namespace

int tuning(Knob k) { return knobs().v[k].load(std::memory_order_relaxed); }

}  // namespace ds

using namespace ds;

extern "C" ds_status ds_set_tuning(const char *name, int32_t value)
{
    if (!name) return fail(DS_ERR_NULL_POINTER, "name must not be NULL");
    const int i = find(name);
    if (i < 0) return fail(DS_ERR_INVALID_ARG, "unknown tuning knob '%s'", name);
    knobs().v[i].store(value < 0 ? -1 : value, std::memory_order_relaxed);
    return ok();
}

extern "C" ds_status ds_get_tuning(const char *name, int32_t *value)
{
    if (!name || !value) return fail(DS_ERR_NULL_POINTER, "name and value must not be NULL");
    const int i = find(name);
    if (i < 0) return fail(DS_ERR_INVALID_ARG, "unknown tuning knob '%s'", name);
    *value = knobs().v[i].load(std::memory_order_relaxed);
    return ok();
}
