// Register-resident row shapes of the read-only row passes (the forward-only
// log-probabilities and the vocabulary shard statistics): one workgroup of
// BLOCK lanes per row, CH 16-byte chunks per lane, the row read once.
//
// These passes read 2V bytes and write a few per row, so unlike the fused
// kernel (which also writes 2V) they run fastest with most of every lane's
// slots full: from 4096 to 9728 chunks per row (32768-77824 columns)
// 512-lane workgroups beat the 1024 x 8 / 1024 x 12 shapes (37984 columns:
// 0.80-0.83 of 8 TB/s against 0.62; 75968: 0.85-0.875 against 0.81), and
// 512 x 5 beats 256 x 12 just above 2048 chunks; 256 x 12 and 256 x 16 stay
// best from 2560 to 4096 chunks.
//
// Each entry serves the rows longer than the entry before it covers
// (block * ch chunks); SAFE is that cover divided by the entry's block,
// rounded down, so its leading SAFE slots hold a chunk of the row in every
// lane.  X(BLOCK, CH, SAFE) is applied to every entry in order.
#pragma once

#include <stdint.h>

#define LEAP_READ_ONLY_SHAPES(X)                                                     \
    X(64, 1, 0) X(64, 2, 1) X(64, 4, 2) X(64, 8, 4) X(256, 4, 2) X(256, 8, 4)        \
    X(512, 5, 4) X(256, 12, 10) X(256, 16, 12) X(512, 10, 8) X(512, 12, 10)           \
    X(512, 16, 12) X(512, 19, 16) X(1024, 12, 9) X(1024, 16, 12) X(1024, 19, 16)      \
    X(1024, 20, 19) X(1024, 24, 20)

namespace leap {
namespace row {

struct ReadOnlyShape {
    int block, ch, safe;
};

#define LEAP_RO_SHAPE_ENTRY(B, C, S) ReadOnlyShape{B, C, S},
constexpr ReadOnlyShape kReadOnlyShapes[] = {LEAP_READ_ONLY_SHAPES(LEAP_RO_SHAPE_ENTRY)};
#undef LEAP_RO_SHAPE_ENTRY
constexpr int kNumReadOnlyShapes = sizeof(kReadOnlyShapes) / sizeof(kReadOnlyShapes[0]);

// Every entry covers more than the one before it, and its SAFE leading slots
// lie inside the shortest row it serves.
constexpr bool read_only_shapes_ordered() {
    int64_t prev = 0;
    for (int i = 0; i < kNumReadOnlyShapes; ++i) {
        const ReadOnlyShape s = kReadOnlyShapes[i];
        const int64_t cover = static_cast<int64_t>(s.block) * s.ch;
        if (cover <= prev || static_cast<int64_t>(s.safe) * s.block > prev || s.safe > s.ch)
            return false;
        prev = cover;
    }
    return true;
}
static_assert(read_only_shapes_ordered(), "read-only row shapes out of order");

// Index of the smallest entry whose chunks cover a row of V columns; -1 when
// the row needs the streaming form.
inline int pick_read_only_shape(int V) {
    const int64_t nchunks = (static_cast<int64_t>(V) + 7) / 8;
    for (int i = 0; i < kNumReadOnlyShapes; ++i)
        if (static_cast<int64_t>(kReadOnlyShapes[i].block) * kReadOnlyShapes[i].ch >= nchunks)
            return i;
    return -1;
}

}  // namespace row
}  // namespace leap
