// tags.h -- step tags of the persistent trainer's exchange words (host side).
//
// Every exchange word carries the 32-bit tag of the step that wrote it; a
// reader takes a word only when its tag equals the current step's. A launch
// of S steps uses tags base .. base + S - 1; the next launch of the same
// context starts at base + S + 2, so no tag of one launch can be read as
// current by the next. Tag 0 is never used: it is what cleared words and
// loads past the end of a buffer return. A tag range that would leave 32 bits
// is never used either: before such a launch the exchange buffers are cleared
// to tag 0 (on the context's stream, after every earlier launch) and the
// tags restart at 1. No HIP dependency, so the arithmetic is testable on the
// host.
#pragma once

#include <stdint.h>

namespace mlp {

struct TagPlan {
    uint32_t base;   // tag of the launch's first step
    uint32_t next;   // tag base of the context's next launch
    bool clear;      // clear the exchange words before this launch
};

// steps: SGD steps of the launch, 1 <= steps < 2^30.
inline TagPlan plan_tags(uint32_t base, int64_t steps) {
    TagPlan p;
    p.clear = false;
    if (base < 1) {                       // a fresh or corrupted base
        base = 1;
        p.clear = true;
    }
    const uint64_t end = (uint64_t)base + (uint64_t)steps + 2u;   // next launch's base
    if (end > 0xFFFFFFFFull) {
        base = 1;
        p.clear = true;
    }
    p.base = base;
    p.next = (uint32_t)((uint64_t)base + (uint64_t)steps + 2u);
    return p;
}

}  // namespace mlp
