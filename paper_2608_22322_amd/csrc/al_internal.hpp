// Launch descriptors and launcher entry points shared between the C ABI
// (al_api.cpp) and the kernel translation units. Not a public header.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "al_device.hpp"

namespace al {

// ------------------------------------------------------------------ AdamW
// One launch covers the whole tensor list: the descriptors live in device
// memory (the caller's workspace), written there on the stream by a copy
// kernel that carries up to kAdamWCopyBatch of them in its arguments.
struct AdamWDesc {
    float* p;
    const void* g;
    void* m;
    float* ms;  // UF8 absmax per 256-element block (unused for FP32 m)
    void* v;
    float* vm;  // AL {l_min, delta} per block (unused for FP32 v)
    int64_t n;
    int64_t tile_begin;  // first chunk of this tensor within the launch
};

struct ApolloDesc;

struct AdamWLaunch {
    double beta1, omb1, beta2, omb2;  // state EMA coefficients (binary64)
    float step_size;                  // lr / (1 - beta1^t)
    float inv_sqrt_bc2;               // 1 / sqrt(1 - beta2^t)
    float eps;
    float decay;                      // 1 - lr * weight_decay
    float v_floor;                    // l_floor of the second-moment code
    const AdamWDesc* D;               // nt descriptors, ascending tile_begin (device memory)
    const int64_t* tb;                // D[i].tile_begin again, packed (the chunk -> tensor search)
    int32_t nt;
    int64_t total_tiles;
    int64_t chunk_base;  // first chunk of this launch (one wave per chunk)
    // APOLLO's moments on the projected gradient at rank 256 (launch_adamw with
    // apollo set): descriptor i is the projected tensor of apollo[i]; there is
    // no parameter stream, and each 256-element sub-tile (one channel) yields
    // the channel scale ||Rt_c|| / (||R_c|| + 1e-8) into apollo[i].s and
    // s_c^2 gn2_c into apollo[i].sg, Rt being the step's direction (the
    // parameter output from zero with lr 1)
    const ApolloDesc* apollo;
};

// Descriptors per copy launch: 60 x 64 bytes keep the argument segment under
// 4 KB.
constexpr int kAdamWCopyBatch = 60;

// Device bytes of the descriptor table of nt tensors (descriptors, then the
// packed chunk offsets), each part 256-byte aligned.
size_t adamw_table_bytes(int64_t nt);
// Copy `count` descriptors (host array) to entries offset.. of an nt-entry
// table at `table`, on the stream.
hipError_t adamw_write_batch(const AdamWDesc* host, int count, int offset, void* table, int64_t nt, hipStream_t s);
// Point a.D / a.tb / a.nt at an nt-entry table.
void adamw_bind_table(void* table, int64_t nt, AdamWLaunch& a);
// Write nt descriptors (host array) into a table at `table` on the stream and
// bind it.
hipError_t adamw_write_table(const AdamWDesc* host, int nt, void* table, AdamWLaunch& a, hipStream_t s);

// The allocation-free AdamW entry point keeps its table in a fixed device
// array of kAdamWScratchBytes (room for kAdamWStaticTensors descriptors) per
// GPU; adamw_static_table returns its device address on the current device
// (looked up once per device).
constexpr int kAdamWStaticTensors = 4096;
constexpr size_t kAdamWScratchBytes = 4096 * 64 + 4096 * 8;  // 288 KiB
constexpr int kMaxDevices = 64;
hipError_t adamw_static_table(void** table);

// Elements per tile: max(block of v, 256).
int adamw_tile_elems(int v_codec, int v_block);
hipError_t launch_adamw(const AdamWLaunch& a, int grad_dtype, int m_codec, int v_codec, int v_block,
                        hipStream_t s, bool apollo = false);

// ------------------------------------------------------------------ codec
hipError_t launch_quantize(int codec, const float* x, int64_t n, int block, float log_floor, void* codes,
                           float* meta, int grid_cap, hipStream_t s);
hipError_t launch_dequantize(int codec, const void* codes, const float* meta, int64_t n, int block,
                             float* out, int grid_cap, hipStream_t s);

hipError_t launch_diag_stream(int mode, float* p, const uint16_t* g, uint8_t* m, uint8_t* v, int64_t n,
                              hipStream_t s);
constexpr int kDiffNormParts = 1024;  // workgroup partials of al_diff_norms (4 doubles each)
hipError_t launch_diff_norms(const float* a, const float* b, int64_t n, double* out, hipStream_t s);
hipError_t launch_diag_math(int fn, const double* x, int64_t n, double* out, int grid_cap, hipStream_t s);

// ---------------------------------------------------- synthetic input fill
hipError_t launch_synth_normal(void* out, int out_bf16, int64_t n, uint64_t key, float scale,
                               uint64_t mask_key, uint64_t mask_threshold, int grid_cap, hipStream_t s);


// ------------------------------------------------------ factored optimizers
// One descriptor per tensor, held in the caller's workspace (written there by
// a device-side copy from the kernel arguments). 2-D tensors (rows > 1) come
// first, then 1-D tensors. Per-tensor workspace regions: column partial sums
// [nru][cols] and row partial sums [ncu][rows] as double-double pairs, the
// reconstruction factors (binary64), fp32 staging for the vector encodes and
// a scalar slot (the clip divisor).
struct FacDesc {
    float* p;
    const void* g;
    int64_t rows, cols;
    void* v;
    float* vm;
    void* vr;
    float* vrm;
    void* vc;
    float* vcm;
    void* m;
    float* mm;
    void* cr;
    float* crm;
    void* cc;
    float* ccm;
    double* colpart;  // [nru][cols] (hi, lo)
    double* rowpart;  // [ncu][rows] (hi, lo)
    double* rfac;     // (R_i / mean R)^-1/2
    double* cfac;     // C_j^-1/2
    double* sr;       // CAME confidence factors
    double* sc;
    float* rtmp;      // staging: R (2-D) or V (1-D)
    float* ctmp;      // staging: C (2-D) or momentum (1-D)
    double* scal;     // [0] = clip divisor max(1, RMS / d)
    double* rsum;     // (hi, lo) per block of the row factor: partial sums of R (or R')
    int64_t unit_begin;   // first 256x256 unit of this tensor (2-D)
    int64_t chunk_begin;  // first 1024-element chunk of this tensor (2-D, cols not a multiple of 256)
    int64_t blk_begin[2];  // first code block of this tensor's R then C (role 0: V, role 1: confidence)
    int32_t nru, ncu;     // units along rows / columns
    int32_t pad_;
};

constexpr int kFacCopyBatch = 16;
struct FacDescBatch {
    int32_t count, offset;
    FacDesc d[kFacCopyBatch];
};

struct FacArgs {
    const FacDesc* D;
    double* rmspart;      // [total_units] (hi, lo): partial sums of u^2
    int32_t n2, n1;       // 2-D tensors, 1-D tensors (D[n2 .. n2 + n1))
    int64_t total_units, total_chunks;
    // units [0, whole_units) belong to the tensors listed first, whose rows and
    // columns are both multiples of 256 (every unit a full 256x256 tile)
    int64_t whole_units;
    int64_t total_blk[2];  // code blocks over all 2-D tensors' R and C, per role
    double beta, omb;     // second-moment EMA: Adafactor beta2_t / CAME beta2, and 1 - beta
    double beta1, omb1;   // CAME momentum
    double beta3, omb3;   // CAME confidence
    double eps1, eps2, lr, decay, clip_d;
    int32_t v_codec, v_block, c_codec, c_block, m_codec, m_block;
    float v_floor, c_floor;
    int32_t exact_all;  // recompute every factored mean exactly (AL_FLAG_EXACT_SUMS)
    Exp2Coef cf;
};

hipError_t launch_diag_levels(int kind, const float* meta, int64_t nblocks, double* out, int grid_cap, hipStream_t s);

hipError_t fac_copy_desc(const FacDesc* host, int count, FacDesc* dev, hipStream_t s);
hipError_t launch_fac_marg_g2(const FacArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_fac_fin(const FacArgs& a, int role, int grad_dtype, hipStream_t s);
hipError_t launch_fac_rms(const FacArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_fac_clip(const FacArgs& a, hipStream_t s);
hipError_t launch_ada_apply(const FacArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_ada_vec1d(const FacArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_came_res(const FacArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_came_apply(const FacArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_came_vec1d(const FacArgs& a, int grad_dtype, hipStream_t s);

// ------------------------------------------------------------------ APOLLO
// One descriptor per projected tensor, held in the caller's workspace. A
// tensor has C channels of L inputs (A = G or G^T as C x L) and rank r; its
// workspace regions hold R and Rt (C x r fp32, channel-major) and per-channel
// binary64 sums.
constexpr int kApolloTileCh = 32;  // channels per projection workgroup
struct ApolloDesc {
    float* p;
    const void* g;
    const float* proj;   // L x r
    float* norm_state;   // limiter state (1 float), or NULL
    float* R;            // C x r: fl32(A Pi)
    float* Rt;           // C x r: the AdamW direction on R (written negated by the AdamW kernel)
    double* gn2;         // C: sum over the channel of g^2
    double* s;           // C: channel scale
    double* sg;          // C: s_c^2 gn2_c
    double* lam;         // [0]: limiter divisor
    int64_t rows, cols, C, L;
    int64_t tile_begin;  // first projection tile (kApolloTileCh channels)
    int64_t chan_begin;  // first channel over the list
    int64_t unit_begin;  // first 256x256 update unit
    int32_t right;       // channels are rows (rows >= cols)
    int32_t nru, ncu;
    int32_t whole;       // rows and columns multiples of 256 (the update takes the streaming chunk layout)
};

constexpr int kApolloCopyBatch = 16;
struct ApolloDescBatch {
    int32_t count, offset;
    ApolloDesc d[kApolloCopyBatch];
};

struct ApolloArgs {
    const ApolloDesc* D;
    int32_t nt, rank;
    int32_t any_whole, any_ragged;  // some tensors are (are not) made of whole 256x256 units
    int64_t total_tiles, total_chans, total_units;
    double lr, decay, gamma;
    int64_t step;
};

hipError_t apollo_copy_desc(const ApolloDesc* host, int count, ApolloDesc* dev, hipStream_t s);
hipError_t launch_apollo_proj(const ApolloArgs& a, int grad_dtype, hipStream_t s);
hipError_t launch_apollo_scale(const ApolloArgs& a, hipStream_t s);
hipError_t launch_apollo_norm(const ApolloArgs& a, hipStream_t s);
hipError_t launch_apollo_update(const ApolloArgs& a, int grad_dtype, hipStream_t s);

// Taylor coefficients of the binary64 exp2 used by every decode.
const Exp2Coef& exp2_coef();

// Compute units of the current device (cached per device).
int device_cu_count();

}  // namespace al
