// Internal interface between the C ABI layer (rf_abi.cpp) and the kernel
// launchers (*.hip). Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rhymeflow.h"

namespace rf {

constexpr int kMaxFrames = RF_MAX_FRAMES;

// Keyframe-query attention launch description. Frame ids travel by value in
// the kernel arguments.
struct AttnParams {
    const void *q;
    const void *k;
    const void *v;
    void *out;
    int64_t S;        // key/value tokens = T * N
    int64_t N;        // tokens per frame
    int32_t M;        // keyframes
    int32_t heads;
    int32_t head_dim;
    int32_t dtype;    // RF_BF16 or RF_F32
    int32_t kf[kMaxFrames];
};

hipError_t launch_attention(const AttnParams &p, hipStream_t stream);

struct ProjParams {
    const void *latents;
    void *out;
    int64_t plane;     // Hl * Wl elements
    int32_t B, C, T;
    int32_t dtype;
    int32_t skip_keyframes;   // out aliases slot 1: leave keyframe planes alone
    float alpha;
    uint8_t is_key[kMaxFrames];
};

hipError_t launch_projection(const ProjParams &p, hipStream_t stream);

struct FrameCopyParams {
    const void *src;
    void *dst;
    int64_t frame_bytes;      // rows_per_frame * row_bytes
    int32_t M;
    int32_t scatter;          // 0: full -> compact, 1: compact -> full
    int32_t ids[kMaxFrames];
};

hipError_t launch_frame_copy(const FrameCopyParams &p, hipStream_t stream);

}  // namespace rf
