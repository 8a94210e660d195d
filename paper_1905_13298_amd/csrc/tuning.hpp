// Tuning overrides of the kernel choices. They change which kernel variant,
// wave split, block order or load depth a call or a plan uses, never its
// results. Each starts from the environment variable of the same name, read
// once when the library is loaded; ds_set_tuning changes it afterwards (tests
// and measurements). -1 means "unset": the library's own choice.
#pragma once

namespace ds {

enum Knob {
    kForceVariant,   // DS_FORCE_VARIANT: 0 one-thread-per-output kernel, 8 tiled with 8 pixels per lane
    kJitWsplit,      // DS_JIT_WSPLIT: waves per 64 pixels in a plan (1, 2, 4, 8, 16)
    kJitSlots,       // DS_JIT_SLOTS: loads in flight per wave in a plan
    kJitMap,         // DS_JIT_MAP: 96 = the 96-register code for one-tap layers too
    kJitGroupTiles,  // DS_JIT_GROUP_TILES: pixel tiles per group of the grouped block order
    kJitOrder,       // DS_JIT_ORDER: 0 grouped, 1 tile-major, 2 XCD-local tile-major
    kJitTn,          // DS_JIT_TN: output channels per code segment in a plan (16, 32, 64)
    kJitPgroups,     // DS_JIT_PGROUPS: groups of 64 pixels per workgroup in a plan (1, 2, 4)
    kRowsBatch,      // DS_ROWS_BATCH: batch rows per workgroup of the small-batch LinearShift (1, 2, 4, 8)
    kJitTranspose,   // DS_JIT_TRANSPOSE: LinearShift plans on x^T: 0 never, 1 from batch 2 (default: batch >= 32)
    kKnobs
};

// Current value of a knob (-1 when unset). Lock-free; safe from any thread.
int tuning(Knob k);

}  // namespace ds
