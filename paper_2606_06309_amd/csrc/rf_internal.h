// Internal interface between the C ABI layer (rf_abi.cpp) and the kernel
// launchers (*.hip). Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rhymeflow.h"

namespace rf {

constexpr int kMaxFrames = RF_MAX_FRAMES;

// Compute units and XCDs (each with its own L2) of the current device, queried
// once per device and kept.
struct DeviceGeometry {
    int32_t cus;
    int32_t xcds;
};

hipError_t device_geometry(DeviceGeometry *out);

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
    // 0: keys are all S tokens; > 0: only the tokens of frames kvf[0..n_kv)
    int32_t n_kv;
    int32_t kvf[kMaxFrames];
    // cache form (bf16): every frame walked; frame f with cslot[f] >= 0 takes
    // the projection of store slots (cslot & 0xffff, cslot >> 16) with weight
    // calpha[f] as its keys and values
    int32_t cache_form;
    const void *store;
    int32_t cslot[kMaxFrames];
    float calpha[kMaxFrames];
    // optional workspace for the split-key tail (NULL: no split)
    void *ws;
    int64_t ws_bytes;
    // the device the launch runs on (bf16: the split plan and the XCD mapping)
    DeviceGeometry geo;
};

// How the bf16 attention of Mq query rows is cut on a device of `cus` compute
// units: n_direct whole tiles, then n_tail tiles split into `split` parts of
// kv_per_split key tiles (split = 0: no split), needing ws_bytes of workspace.
struct AttnSplit {
    int64_t n_tiles;
    int64_t n_direct;
    int64_t n_tail;
    int64_t split;
    int64_t kv_per_split;
    int64_t ws_bytes;
};

// walk_frames > 0: the key loop walks that many whole frames in frame-aligned
// tiles (the cache form) while the number of parts is chosen as for n_kv.
AttnSplit attention_split(int64_t Mq, int32_t heads, int32_t head_dim, int64_t N, int64_t S, int32_t n_kv,
                          int32_t cus, int32_t walk_frames = 0);


hipError_t launch_attention(const AttnParams &p, hipStream_t stream);

// Static split-tail scratch of the allocation-free attention entry point (a
// file-scope device array in rf_noalloc.hip): its size, and its device address
// on the current device (looked up once per device).
constexpr int64_t kAttentionScratchBytes = int64_t(160) << 20;
hipError_t attention_scratch(void **out);

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

// Copies of whole frames: block src_idx[m] of src to block dst_idx[m] of dst,
// m < M, each block frame_bytes long (gather: src_idx = ids, dst_idx = m;
// scatter: the reverse; rolling-cache store: frame -> cache slot).
struct FrameCopyParams {
    const void *src;
    void *dst;
    int64_t frame_bytes;      // rows_per_frame * row_bytes
    int32_t M;
    int32_t src_idx[kMaxFrames];
    int32_t dst_idx[kMaxFrames];
};

hipError_t launch_frame_copy(const FrameCopyParams &p, hipStream_t stream);

// Rolling-cache projection (App. B.2): for entry m, frame block dst[m] of both
// k and v receives fmaf(alpha[m], after, (1 - alpha[m]) * before) of store
// slots before[m] and after[m].
struct CacheProjParams {
    const void *store;
    void *k;
    void *v;
    int64_t frame_bytes;
    int32_t n;
    int32_t dtype;
    int16_t before[kMaxFrames];
    int16_t after[kMaxFrames];
    uint8_t dst[kMaxFrames];
    float alpha[kMaxFrames];
};

hipError_t launch_cache_projection(const CacheProjParams &p, hipStream_t stream);

// Frame cosine similarity: blocking of the frame Gram matrix over feature
// chunks (shared by the workspace query and the launcher).
struct SimGeometry {
    int32_t Tp;               // frames rounded up to a multiple of 4
    int32_t NB;               // 4-frame blocks
    int32_t NBP;              // block pairs (bi <= bj)
    int32_t L;                // feature elements per chunk
    int64_t chunks_per_plane;
    int64_t n_chunks;         // per batch element: C * chunks_per_plane
    int64_t run;              // consecutive chunks one workgroup accumulates
    int64_t n_runs;           // workgroups (partial Gram blocks) per batch element
    int64_t workspace_bytes;  // B * n_runs * NBP * 16 doubles
};

SimGeometry similarity_geometry(int32_t B, int32_t C, int32_t T, int64_t plane);

struct SimParams {
    const void *latents;
    double *sim;
    double *workspace;
    int64_t plane;            // H * W
    int32_t B, C, T;
    int32_t dtype;
};

hipError_t launch_similarity(const SimParams &p, hipStream_t stream);

// Device probes (measurement support): threads per workgroup of the matrix and
// LDS probes, and of the HBM read probe.
constexpr int kProbeThreads = 256;
constexpr int kHbmThreads = 1024;
hipError_t launch_mfma_probe(const void *ops, int32_t workgroups, int32_t rounds, float *sink,
                             hipStream_t stream);
hipError_t launch_lds_read_probe(int32_t workgroups, int32_t rounds, int32_t width, uint32_t *sink,
                                 uint64_t *ticks, hipStream_t stream);
hipError_t launch_hbm_read_probe(const void *src, int64_t bytes, int32_t workgroups, uint32_t *sink,
                                 hipStream_t stream);

}  // namespace rf
