// C ABI of libal.so: argument validation (on the host, before any HIP call),
// storage accounting, scalar precompute in binary64, and launches on the
// caller's stream. See include/al.h for the contract of each entry point.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "../../include/al.h"
#include "../../include/al_synth.h"
#include "al_internal.hpp"

namespace {

thread_local char g_err[512] = "";

al_status fail(al_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return s;
}

al_status hip_fail(hipError_t e, const char* what) {
    return fail(AL_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_block(int32_t b) { return b == 64 || b == 128 || b == 256 || b == 512 || b == 1024 || b == 2048; }

bool valid_codec(int32_t c) { return c >= AL_CODEC_FP32 && c <= AL_CODEC_UF8; }

bool is_fin(double x) { return std::isfinite(x); }

int64_t nblocks(int64_t n, int32_t b) { return (n + b - 1) / b; }

// Validate a state spec for a role: `allowed` is a bit mask of codecs.
al_status check_spec(const al_state_spec& s, unsigned allowed, const char* role) {
    if (!valid_codec(s.codec) || !((allowed >> s.codec) & 1u))
        return fail(AL_EINVAL, "%s: codec %d not allowed for this state", role, s.codec);
    if (s.codec != AL_CODEC_FP32 && !valid_block(s.block))
        return fail(AL_EINVAL, "%s: block %d must be 64, 128, 256, 512, 1024 or 2048", role, s.block);
    if ((s.codec == AL_CODEC_AL8 || s.codec == AL_CODEC_AL16) && !std::isfinite(s.log_floor))
        return fail(AL_EINVAL, "%s: log_floor must be finite", role);
    return AL_OK;
}

// A state slot: codes non-NULL and aligned; metadata required iff quantized.
al_status check_state(const void* codes, const float* meta, const al_state_spec& s, int64_t n, const char* role,
                      int i) {
    if (n == 0) return AL_OK;
    if (!codes) return fail(AL_EINVAL, "tensor %d: %s buffer is NULL", i, role);
    if (!aligned16(codes)) return fail(AL_EALIGN, "tensor %d: %s buffer not 16-byte aligned", i, role);
    if (s.codec != AL_CODEC_FP32) {
        if (!meta) return fail(AL_EINVAL, "tensor %d: %s metadata is NULL", i, role);
        if (!aligned16(meta)) return fail(AL_EALIGN, "tensor %d: %s metadata not 16-byte aligned", i, role);
    }
    return AL_OK;
}

al_status check_unused(const void* a, const void* b, const char* role, int i) {
    if (a || b) return fail(AL_EINVAL, "tensor %d: %s must be NULL for this path", i, role);
    return AL_OK;
}

al_status check_shape(const al_tensor& t, int i, int64_t* n_out) {
    if (t.rows < 0 || t.cols < 0) return fail(AL_EINVAL, "tensor %d: negative shape", i);
    if (t.rows > 0 && t.cols > (int64_t(1) << 62) / t.rows) return fail(AL_EINVAL, "tensor %d: shape overflows", i);
    const int64_t n = t.rows * t.cols;
    if (n > 0) {
        if (!t.param || !t.grad) return fail(AL_EINVAL, "tensor %d: param or grad is NULL", i);
        if (!aligned16(t.param) || !aligned16(t.grad))
            return fail(AL_EALIGN, "tensor %d: param or grad not 16-byte aligned", i);
    }
    *n_out = n;
    return AL_OK;
}

// ------------------------------------------------------ factored-path plan
const al_state_spec kNoSpec = {AL_CODEC_FP32, 256, 0.0f};

al_status check_adafactor_cfg(const al_adafactor_cfg* cfg) {
    if (!cfg) return fail(AL_EINVAL, "adafactor: cfg is NULL");
    if (cfg->grad_dtype != AL_DTYPE_F32 && cfg->grad_dtype != AL_DTYPE_BF16)
        return fail(AL_EINVAL, "adafactor: grad_dtype %d", cfg->grad_dtype);
    if (!is_fin(cfg->lr) || cfg->lr < 0 || !is_fin(cfg->eps1) || cfg->eps1 < 0 || !is_fin(cfg->clip_threshold) ||
        !(cfg->clip_threshold > 0) || !is_fin(cfg->decay_rate) || cfg->decay_rate > 0 ||
        !is_fin(cfg->weight_decay) || cfg->weight_decay < 0)
        return fail(AL_EINVAL, "adafactor: hyperparameters out of range");
    if (cfg->flags & ~AL_FLAG_EXACT_SUMS) return fail(AL_EINVAL, "adafactor: unknown flags 0x%x", cfg->flags);
    return check_spec(cfg->v, (1u << AL_CODEC_FP32) | (1u << AL_CODEC_AL8) | (1u << AL_CODEC_AL16), "v");
}

al_status check_came_cfg(const al_came_cfg* cfg) {
    if (!cfg) return fail(AL_EINVAL, "came: cfg is NULL");
    if (cfg->grad_dtype != AL_DTYPE_F32 && cfg->grad_dtype != AL_DTYPE_BF16)
        return fail(AL_EINVAL, "came: grad_dtype %d", cfg->grad_dtype);
    if (!is_fin(cfg->lr) || cfg->lr < 0 || !is_fin(cfg->eps1) || cfg->eps1 < 0 || !is_fin(cfg->eps2) ||
        cfg->eps2 < 0 || !is_fin(cfg->clip_threshold) || !(cfg->clip_threshold > 0) || !is_fin(cfg->weight_decay) ||
        cfg->weight_decay < 0 || !(cfg->beta1 >= 0 && cfg->beta1 < 1) || !(cfg->beta2 >= 0 && cfg->beta2 < 1) ||
        !(cfg->beta3 >= 0 && cfg->beta3 < 1))
        return fail(AL_EINVAL, "came: hyperparameters out of range");
    if (cfg->flags & ~AL_FLAG_EXACT_SUMS) return fail(AL_EINVAL, "came: unknown flags 0x%x", cfg->flags);
    al_status st;
    const unsigned nonneg = (1u << AL_CODEC_FP32) | (1u << AL_CODEC_AL8) | (1u << AL_CODEC_AL16);
    if ((st = check_spec(cfg->m, (1u << AL_CODEC_FP32) | (1u << AL_CODEC_UF8), "m")) != AL_OK) return st;
    if ((st = check_spec(cfg->v, nonneg, "v")) != AL_OK) return st;
    if ((st = check_spec(cfg->conf, nonneg, "conf")) != AL_OK) return st;
    if (cfg->m.codec == AL_CODEC_UF8 && cfg->m.block != 256)
        return fail(AL_EUNSUPPORTED, "came: UF8 momentum block must be 256 (got %d)", cfg->m.block);
    return AL_OK;
}

al_status check_ws(void* ws, size_t ws_bytes, size_t need, const char* who) {
    if (need == 0) return AL_OK;
    if (!ws) return fail(AL_EWORKSPACE, "%s: workspace is NULL (need %zu bytes)", who, need);
    if (ws_bytes < need) return fail(AL_EWORKSPACE, "%s: workspace %zu bytes < %zu needed", who, ws_bytes, need);
    if (reinterpret_cast<uintptr_t>(ws) & 255u) return fail(AL_EALIGN, "%s: workspace not 256-byte aligned", who);
    return AL_OK;
}

struct FacPlan {
    std::vector<al::FacDesc> desc;  // 2-D tensors first, then 1-D
    int n2 = 0, n1 = 0;
    int64_t total_units = 0, total_chunks = 0, whole_units = 0;
    int64_t total_blk[2] = {0, 0};
    size_t bytes = 0;
    size_t rms_off = 0;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Validate the tensor list and lay out the workspace: descriptor table, RMS
// partials, then per-tensor regions. With ws == NULL only sizes are computed.
al_status fac_plan(const al_tensor* ts, int nt, bool came, const al_state_spec& ms, const al_state_spec& vs,
                   const al_state_spec& cs, char* ws, FacPlan& P) {
    const char* who = came ? "al_came_step" : "al_adafactor_step";
    if (nt < 0) return fail(AL_EINVAL, "%s: nt < 0", who);
    if (nt > 0 && !ts) return fail(AL_EINVAL, "%s: tensors is NULL", who);
    P = FacPlan();
    std::vector<int> twod, oned;
    al_status st;
    for (int i = 0; i < nt; ++i) {
        const al_tensor& t = ts[i];
        int64_t n = 0;
        if ((st = check_shape(t, i, &n)) != AL_OK) return st;
        if (n == 0) continue;
        const bool fac = t.rows > 1;
        if (fac) {
            if ((st = check_state(t.vr, t.vr_meta, vs, t.rows, "vr", i)) != AL_OK) return st;
            if ((st = check_state(t.vc, t.vc_meta, vs, t.cols, "vc", i)) != AL_OK) return st;
            if ((st = check_unused(t.v, t.v_meta, "v (2-D tensor)", i)) != AL_OK) return st;
            if (came) {
                if ((st = check_state(t.cr, t.cr_meta, cs, t.rows, "cr", i)) != AL_OK) return st;
                if ((st = check_state(t.cc, t.cc_meta, cs, t.cols, "cc", i)) != AL_OK) return st;
            } else {
                if ((st = check_unused(t.cr, t.cr_meta, "cr", i)) != AL_OK) return st;
                if ((st = check_unused(t.cc, t.cc_meta, "cc", i)) != AL_OK) return st;
            }
            twod.push_back(i);
        } else {
            if ((st = check_state(t.v, t.v_meta, vs, n, "v", i)) != AL_OK) return st;
            if ((st = check_unused(t.vr, t.vr_meta, "vr (1-D tensor)", i)) != AL_OK) return st;
            if ((st = check_unused(t.vc, t.vc_meta, "vc (1-D tensor)", i)) != AL_OK) return st;
            if ((st = check_unused(t.cr, t.cr_meta, "cr (1-D tensor)", i)) != AL_OK) return st;
            if ((st = check_unused(t.cc, t.cc_meta, "cc (1-D tensor)", i)) != AL_OK) return st;
            oned.push_back(i);
        }
        if (came) {
            if ((st = check_state(t.m, t.m_meta, ms, n, "m", i)) != AL_OK) return st;
        } else {
            if ((st = check_unused(t.m, t.m_meta, "m", i)) != AL_OK) return st;
        }
    }
    // 2-D tensors made of whole 256x256 units first (their units take the
    // streaming kernels' guard-free layout), in list order within each group
    std::stable_partition(twod.begin(), twod.end(),
                          [&](int i) { return ts[i].rows % 256 == 0 && ts[i].cols % 256 == 0; });
    P.n2 = (int)twod.size();
    P.n1 = (int)oned.size();
    const int ntot = P.n2 + P.n1;
    P.desc.resize(ntot);
    for (int k = 0; k < P.n2; ++k) {
        const al_tensor& t = ts[twod[k]];
        al::FacDesc& d = P.desc[k];
        d.nru = (int32_t)((t.rows + 255) / 256);
        d.ncu = (int32_t)((t.cols + 255) / 256);
        d.unit_begin = P.total_units;
        P.total_units += (int64_t)d.nru * d.ncu;
        if (t.rows % 256 == 0 && t.cols % 256 == 0) P.whole_units = P.total_units;
        d.chunk_begin = P.total_chunks;  // chunks only for widths that are not a multiple of 256
        if (t.cols % 256 != 0) P.total_chunks += (t.rows * t.cols + 1023) / 1024;
        const int64_t bv = vs.block, bc = came ? cs.block : vs.block;
        d.blk_begin[0] = P.total_blk[0];
        P.total_blk[0] += (t.rows + bv - 1) / bv + (t.cols + bv - 1) / bv;
        d.blk_begin[1] = P.total_blk[1];
        P.total_blk[1] += (t.rows + bc - 1) / bc + (t.cols + bc - 1) / bc;
    }
    size_t off = align256((size_t)ntot * sizeof(al::FacDesc));
    P.rms_off = off;
    off += align256((size_t)P.total_units * 16);
    auto take = [&](size_t nbytes) -> char* {
        char* ptr = ws ? ws + off : nullptr;
        off += align256(nbytes);
        return ptr;
    };
    for (int k = 0; k < ntot; ++k) {
        const bool fac = k < P.n2;
        const al_tensor& t = ts[fac ? twod[k] : oned[k - P.n2]];
        al::FacDesc& d = P.desc[k];
        d.p = t.param;
        d.g = t.grad;
        d.rows = t.rows;
        d.cols = t.cols;
        d.v = t.v;
        d.vm = t.v_meta;
        d.vr = t.vr;
        d.vrm = t.vr_meta;
        d.vc = t.vc;
        d.vcm = t.vc_meta;
        d.m = t.m;
        d.mm = t.m_meta;
        d.cr = t.cr;
        d.crm = t.cr_meta;
        d.cc = t.cc;
        d.ccm = t.cc_meta;
        if (fac) {
            // (hi, lo) pairs per unit and column / row; whole-unit tensors use the first half
            d.colpart = reinterpret_cast<double*>(take((size_t)d.nru * t.cols * 16));
            d.rowpart = reinterpret_cast<double*>(take((size_t)d.ncu * t.rows * 16));
            d.rfac = reinterpret_cast<double*>(take((size_t)t.rows * 8));
            d.cfac = reinterpret_cast<double*>(take((size_t)t.cols * 8));
            if (came) {
                d.sr = reinterpret_cast<double*>(take((size_t)t.rows * 8));
                d.sc = reinterpret_cast<double*>(take((size_t)t.cols * 8));
            }
            d.rtmp = reinterpret_cast<float*>(take((size_t)t.rows * 4));
            d.ctmp = reinterpret_cast<float*>(take((size_t)t.cols * 4));
            const int64_t bmin = came && cs.block < vs.block ? cs.block : vs.block;
            d.rsum = reinterpret_cast<double*>(take((size_t)((t.rows + bmin - 1) / bmin) * 16));
        } else {
            d.nru = d.ncu = 0;
            const size_t n = (size_t)(t.rows * t.cols);
            d.rtmp = reinterpret_cast<float*>(take(n * 4));
            if (came) d.ctmp = reinterpret_cast<float*>(take(n * 4));
        }
        d.scal = reinterpret_cast<double*>(take(16));
    }
    P.bytes = off;
    return AL_OK;
}

al::FacArgs fac_args(const FacPlan& P, char* ws) {
    al::FacArgs a;
    std::memset(&a, 0, sizeof(a));
    a.D = reinterpret_cast<const al::FacDesc*>(ws);
    a.rmspart = reinterpret_cast<double*>(ws + P.rms_off);
    a.n2 = P.n2;
    a.n1 = P.n1;
    a.total_units = P.total_units;
    a.total_chunks = P.total_chunks;
    a.whole_units = P.whole_units;
    a.total_blk[0] = P.total_blk[0];
    a.total_blk[1] = P.total_blk[1];
    a.cf = al::exp2_coef();
    a.m_block = 256;
    return a;
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ------------------------------------------------------------ APOLLO plan
al_status check_apollo_cfg(const al_apollo_cfg* cfg) {
    if (!cfg) return fail(AL_EINVAL, "apollo: cfg is NULL");
    if (cfg->grad_dtype != AL_DTYPE_F32 && cfg->grad_dtype != AL_DTYPE_BF16)
        return fail(AL_EINVAL, "apollo: grad_dtype %d", cfg->grad_dtype);
    if (cfg->rank != 64 && cfg->rank != 128 && cfg->rank != 256)
        return fail(AL_EINVAL, "apollo: rank %d must be 64, 128 or 256", cfg->rank);
    if (!is_fin(cfg->lr) || cfg->lr < 0 || !is_fin(cfg->eps) || cfg->eps < 0 || !is_fin(cfg->weight_decay) ||
        cfg->weight_decay < 0 || !is_fin(cfg->gamma) || !(cfg->beta1 >= 0 && cfg->beta1 < 1) ||
        !(cfg->beta2 >= 0 && cfg->beta2 < 1))
        return fail(AL_EINVAL, "apollo: hyperparameters out of range");
    al_status st;
    if ((st = check_spec(cfg->m, (1u << AL_CODEC_FP32) | (1u << AL_CODEC_UF8), "m")) != AL_OK) return st;
    if ((st = check_spec(cfg->v, (1u << AL_CODEC_FP32) | (1u << AL_CODEC_AL8) | (1u << AL_CODEC_AL16), "v")) !=
        AL_OK)
        return st;
    if (cfg->m.codec == AL_CODEC_UF8 && cfg->m.block != 256)
        return fail(AL_EUNSUPPORTED, "apollo: UF8 momentum block must be 256 (got %d)", cfg->m.block);
    return AL_OK;
}

struct ApolloPlan {
    std::vector<al::ApolloDesc> desc;
    std::vector<int> idx;  // tensor index of each descriptor (empty tensors are skipped)
    int64_t total_tiles = 0, total_chans = 0, total_units = 0;
    int32_t any_whole = 0, any_ragged = 0;
    size_t adamw_off = 0;  // descriptor table of the AdamW launch over the projected moments
    size_t bytes = 0;
};

// Validate the list and lay out the workspace: descriptor table, then per
// tensor R, Rt (C x rank fp32; no Rt at rank 256, where the AdamW step on R
// reduces the direction into the channel scales itself), gn2, s, sg (C
// doubles) and the limiter slot.
// At rank 256 a channel of R is one 256-element sub-tile of the AdamW step,
// which then forms the channel scales itself (no Rt, no scale pass).
bool apollo_fused(int64_t rank) { return rank == 256; }

al_status apollo_plan(const al_apollo_tensor* ts, int nt, const al_apollo_cfg* cfg, char* ws, ApolloPlan& P) {
    if (nt < 0) return fail(AL_EINVAL, "apollo: nt < 0");
    if (nt > 0 && !ts) return fail(AL_EINVAL, "apollo: tensors is NULL");
    P = ApolloPlan();
    const int64_t r = cfg->rank;
    for (int i = 0; i < nt; ++i) {
        const al_apollo_tensor& t = ts[i];
        if (t.rows < 0 || t.cols < 0) return fail(AL_EINVAL, "tensor %d: negative shape", i);
        if (t.rows > 0 && t.cols > (int64_t(1) << 40) / t.rows) return fail(AL_EINVAL, "tensor %d: shape too large", i);
        if (t.rows * t.cols == 0) continue;
        if (!t.param || !t.grad || !t.proj) return fail(AL_EINVAL, "tensor %d: param, grad or proj is NULL", i);
        if (!aligned16(t.param) || !aligned16(t.grad) || !aligned16(t.proj))
            return fail(AL_EALIGN, "tensor %d: param, grad or proj not 16-byte aligned", i);
        const int64_t C = t.rows >= t.cols ? t.rows : t.cols;
        al_status st;
        if ((st = check_state(t.m, t.m_meta, cfg->m, C * r, "m", i)) != AL_OK) return st;
        if ((st = check_state(t.v, t.v_meta, cfg->v, C * r, "v", i)) != AL_OK) return st;
        if (cfg->gamma > 0) {
            if (!t.norm_state) return fail(AL_EINVAL, "tensor %d: norm_state is NULL (the limiter is on)", i);
            if (!aligned16(t.norm_state)) return fail(AL_EALIGN, "tensor %d: norm_state not 16-byte aligned", i);
        }
        al::ApolloDesc d;
        std::memset(&d, 0, sizeof(d));
        d.p = t.param;
        d.g = t.grad;
        d.proj = t.proj;
        d.norm_state = t.norm_state;
        d.rows = t.rows;
        d.cols = t.cols;
        d.right = t.rows >= t.cols;
        d.C = C;
        d.L = d.right ? t.cols : t.rows;
        d.nru = (int32_t)((t.rows + 255) / 256);
        d.ncu = (int32_t)((t.cols + 255) / 256);
        d.tile_begin = P.total_tiles;
        P.total_tiles += (C + al::kApolloTileCh - 1) / al::kApolloTileCh;
        d.chan_begin = P.total_chans;
        P.total_chans += C;
        d.unit_begin = P.total_units;
        P.total_units += (int64_t)d.nru * d.ncu;
        d.whole = t.rows % 256 == 0 && t.cols % 256 == 0;
        (d.whole ? P.any_whole : P.any_ragged) = 1;
        P.desc.push_back(d);
        P.idx.push_back(i);
    }
    if (P.total_tiles >= (int64_t(1) << 31) || P.total_chans / 4 >= (int64_t(1) << 31) ||
        P.total_units / 4 >= (int64_t(1) << 31))
        return fail(AL_EUNSUPPORTED, "apollo: tensor list too large for one launch");
    size_t off = align256(P.desc.size() * sizeof(al::ApolloDesc));
    auto take = [&](size_t nbytes) -> char* {
        char* ptr = ws ? ws + off : nullptr;
        off += align256(nbytes);
        return ptr;
    };
    for (auto& d : P.desc) {
        d.R = reinterpret_cast<float*>(take((size_t)(d.C * r) * 4));
        d.Rt = apollo_fused(r) ? nullptr : reinterpret_cast<float*>(take((size_t)(d.C * r) * 4));
        d.gn2 = reinterpret_cast<double*>(take((size_t)d.C * 8));
        d.s = reinterpret_cast<double*>(take((size_t)d.C * 8));
        d.sg = reinterpret_cast<double*>(take((size_t)d.C * 8));
        d.lam = reinterpret_cast<double*>(take(16));
    }
    P.adamw_off = off;
    off += al::adamw_table_bytes((int64_t)P.desc.size());
    P.bytes = P.desc.empty() ? 0 : off;
    return AL_OK;
}

}  // namespace

namespace al {

int device_cu_count() {
    static std::mutex mu;
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    std::lock_guard<std::mutex> lk(mu);
    if (cache[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cache[dev] = v;
    }
    return cache[dev];
}

}  // namespace al

extern "C" {

const char* al_version(void) { return "0.1.0 gfx950"; }

const char* al_last_error(void) { return g_err; }

int64_t al_code_bytes(int32_t codec, int64_t n, int32_t block) {
    if (n < 0 || !valid_codec(codec)) return -1;
    if (codec == AL_CODEC_FP32) return 4 * n;
    if (!valid_block(block)) return -1;
    const int64_t padded = nblocks(n, block) * block;
    return codec == AL_CODEC_AL16 ? 2 * padded : padded;
}

int64_t al_meta_floats(int32_t codec, int64_t n, int32_t block) {
    if (n < 0 || !valid_codec(codec)) return -1;
    if (codec == AL_CODEC_FP32) return 0;
    if (!valid_block(block)) return -1;
    return nblocks(n, block) * (codec == AL_CODEC_UF8 ? 1 : 2);
}

int64_t al_state_bytes(int32_t codec, int64_t n, int32_t block) {
    const int64_t c = al_code_bytes(codec, n, block);
    const int64_t m = al_meta_floats(codec, n, block);
    if (c < 0 || m < 0) return -1;
    return c + 4 * m;
}

al_status al_quantize(int32_t codec, const float* x, int64_t n, int32_t block, float log_floor, void* codes,
                      float* meta, void* stream) {
    g_err[0] = 0;
    if (codec != AL_CODEC_AL8 && codec != AL_CODEC_AL16 && codec != AL_CODEC_UF8)
        return fail(AL_EINVAL, "al_quantize: codec %d is not AL8, AL16 or UF8", codec);
    if (n < 0) return fail(AL_EINVAL, "al_quantize: n < 0");
    if (!valid_block(block)) return fail(AL_EINVAL, "al_quantize: block %d invalid", block);
    if (codec != AL_CODEC_UF8 && !std::isfinite(log_floor)) return fail(AL_EINVAL, "al_quantize: log_floor");
    if (n == 0) return AL_OK;
    if (!x || !codes || !meta) return fail(AL_EINVAL, "al_quantize: NULL buffer");
    if (!aligned16(x) || !aligned16(codes) || !aligned16(meta)) return fail(AL_EALIGN, "al_quantize: alignment");
    hipError_t e = al::launch_quantize(codec, x, n, block, log_floor, codes, meta, al::device_cu_count() * 8,
                                       as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_quantize launch");
}

al_status al_dequantize(int32_t codec, const void* codes, const float* meta, int64_t n, int32_t block, float* out,
                        void* stream) {
    g_err[0] = 0;
    if (codec != AL_CODEC_AL8 && codec != AL_CODEC_AL16 && codec != AL_CODEC_UF8)
        return fail(AL_EINVAL, "al_dequantize: codec %d is not AL8, AL16 or UF8", codec);
    if (n < 0) return fail(AL_EINVAL, "al_dequantize: n < 0");
    if (!valid_block(block)) return fail(AL_EINVAL, "al_dequantize: block %d invalid", block);
    if (n == 0) return AL_OK;
    if (!codes || !meta || !out) return fail(AL_EINVAL, "al_dequantize: NULL buffer");
    if (!aligned16(out) || !aligned16(codes) || !aligned16(meta)) return fail(AL_EALIGN, "al_dequantize: alignment");
    hipError_t e = al::launch_dequantize(codec, codes, meta, n, block, out, al::device_cu_count() * 8,
                                         as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_dequantize launch");
}

}  // extern "C"

namespace {

// Validate an AdamW call, count its non-empty tensors and set the launch
// constants (a.total_tiles included). No HIP call.
al_status adamw_check(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, int64_t step, const char* who,
                      int64_t* ndesc, al::AdamWLaunch& a) {
    if (nt < 0) return fail(AL_EINVAL, "%s: nt < 0", who);
    if (nt > 0 && !tensors) return fail(AL_EINVAL, "%s: tensors is NULL", who);
    if (!cfg) return fail(AL_EINVAL, "%s: cfg is NULL", who);
    if (step < 1) return fail(AL_EINVAL, "%s: step must be >= 1", who);
    if (cfg->grad_dtype != AL_DTYPE_F32 && cfg->grad_dtype != AL_DTYPE_BF16)
        return fail(AL_EINVAL, "%s: grad_dtype %d", who, cfg->grad_dtype);
    if (!is_fin(cfg->lr) || cfg->lr < 0 || !is_fin(cfg->eps) || cfg->eps < 0 || !is_fin(cfg->weight_decay) ||
        cfg->weight_decay < 0 || !(cfg->beta1 >= 0 && cfg->beta1 < 1) || !(cfg->beta2 >= 0 && cfg->beta2 < 1))
        return fail(AL_EINVAL, "%s: hyperparameters out of range", who);
    al_status st;
    if ((st = check_spec(cfg->m, (1u << AL_CODEC_FP32) | (1u << AL_CODEC_UF8), "m")) != AL_OK) return st;
    if ((st = check_spec(cfg->v, (1u << AL_CODEC_FP32) | (1u << AL_CODEC_AL8) | (1u << AL_CODEC_AL16), "v")) !=
        AL_OK)
        return st;
    if (cfg->m.codec == AL_CODEC_UF8 && cfg->m.block != 256)
        return fail(AL_EUNSUPPORTED, "%s: UF8 momentum block must be 256 (got %d)", who, cfg->m.block);

    std::memset(&a, 0, sizeof(a));
    *ndesc = 0;
    const int T = al::adamw_tile_elems(cfg->v.codec, cfg->v.block);
    for (int i = 0; i < nt; ++i) {
        const al_tensor& t = tensors[i];
        int64_t n = 0;
        if ((st = check_shape(t, i, &n)) != AL_OK) return st;
        if ((st = check_state(t.m, t.m_meta, cfg->m, n, "m", i)) != AL_OK) return st;
        if ((st = check_state(t.v, t.v_meta, cfg->v, n, "v", i)) != AL_OK) return st;
        if ((st = check_unused(t.vr, t.vr_meta, "vr", i)) != AL_OK) return st;
        if ((st = check_unused(t.vc, t.vc_meta, "vc", i)) != AL_OK) return st;
        if ((st = check_unused(t.cr, t.cr_meta, "cr", i)) != AL_OK) return st;
        if ((st = check_unused(t.cc, t.cc_meta, "cc", i)) != AL_OK) return st;
        if (n == 0) continue;
        ++*ndesc;
        a.total_tiles += (n + T - 1) / T;
    }
    const double bc1 = 1.0 - std::pow(cfg->beta1, (double)step);
    const double bc2 = 1.0 - std::pow(cfg->beta2, (double)step);
    a.beta1 = cfg->beta1;
    a.omb1 = 1.0 - cfg->beta1;
    a.beta2 = cfg->beta2;
    a.omb2 = 1.0 - cfg->beta2;
    a.step_size = (float)(cfg->lr / bc1);
    a.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
    a.eps = (float)cfg->eps;
    a.decay = (float)(1.0 - cfg->lr * cfg->weight_decay);
    a.v_floor = cfg->v.log_floor;
    return AL_OK;
}

// Write the descriptors of a validated list into an ndesc-entry table, a copy
// launch per kAdamWCopyBatch of them (built in a stack buffer: no heap), bind
// the table and launch the step.
al_status adamw_run(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, int64_t ndesc, void* table,
                    al::AdamWLaunch& a, hipStream_t s, const char* who) {
    const int T = al::adamw_tile_elems(cfg->v.codec, cfg->v.block);
    al::AdamWDesc batch[al::kAdamWCopyBatch];
    int nb = 0, off = 0;
    int64_t tile = 0;
    hipError_t e;
    for (int i = 0; i < nt; ++i) {
        const al_tensor& t = tensors[i];
        const int64_t n = t.rows * t.cols;
        if (n == 0) continue;
        al::AdamWDesc& d = batch[nb++];
        d.p = t.param;
        d.g = t.grad;
        d.m = t.m;
        d.ms = t.m_meta;
        d.v = t.v;
        d.vm = t.v_meta;
        d.n = n;
        d.tile_begin = tile;
        tile += (n + T - 1) / T;
        if (nb == al::kAdamWCopyBatch) {
            if ((e = al::adamw_write_batch(batch, nb, off, table, ndesc, s)) != hipSuccess) return hip_fail(e, who);
            off += nb;
            nb = 0;
        }
    }
    if (nb > 0 && (e = al::adamw_write_batch(batch, nb, off, table, ndesc, s)) != hipSuccess) return hip_fail(e, who);
    al::adamw_bind_table(table, ndesc, a);
    if ((e = al::launch_adamw(a, cfg->grad_dtype, cfg->m.codec, cfg->v.codec, cfg->v.block, s)) != hipSuccess)
        return hip_fail(e, who);
    return AL_OK;
}

}  // namespace

extern "C" {

al_status al_adamw_workspace_bytes(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, size_t* bytes) {
    g_err[0] = 0;
    if (!bytes) return fail(AL_EINVAL, "al_adamw_workspace_bytes: bytes is NULL");
    *bytes = 0;
    int64_t ndesc = 0;
    al::AdamWLaunch a;
    const al_status st = adamw_check(tensors, nt, cfg, 1, "al_adamw_workspace_bytes", &ndesc, a);
    if (st != AL_OK) return st;
    *bytes = al::adamw_table_bytes(ndesc);
    return AL_OK;
}

al_status al_adamw_step(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, int64_t step, void* ws,
                        size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    int64_t ndesc = 0;
    al::AdamWLaunch a;
    al_status st = adamw_check(tensors, nt, cfg, step, "al_adamw_step", &ndesc, a);
    if (st != AL_OK) return st;
    if (ndesc == 0) return AL_OK;
    if ((st = check_ws(ws, ws_bytes, al::adamw_table_bytes(ndesc), "al_adamw_step")) != AL_OK) return st;
    return adamw_run(tensors, nt, cfg, ndesc, ws, a, as_stream(stream), "al_adamw_step launch");
}

al_status al_adamw_step_noalloc(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, int64_t step,
                                void* stream) {
    g_err[0] = 0;
    int64_t ndesc = 0;
    al::AdamWLaunch a;
    al_status st = adamw_check(tensors, nt, cfg, step, "al_adamw_step_noalloc", &ndesc, a);
    if (st != AL_OK) return st;
    if (ndesc == 0) return AL_OK;
    if (ndesc > al::kAdamWStaticTensors)
        return fail(AL_EUNSUPPORTED,
                    "al_adamw_step_noalloc: %lld non-empty tensors exceed its fixed table of %d "
                    "(use al_adamw_step with a workspace)",
                    (long long)ndesc, al::kAdamWStaticTensors);
    void* table = nullptr;
    const hipError_t e = al::adamw_static_table(&table);
    if (e != hipSuccess) return hip_fail(e, "al_adamw_step_noalloc: static table address");
    return adamw_run(tensors, nt, cfg, ndesc, table, a, as_stream(stream), "al_adamw_step_noalloc launch");
}

al_status al_apollo_workspace_bytes(const al_apollo_tensor* tensors, int32_t nt, const al_apollo_cfg* cfg,
                                    size_t* bytes) {
    g_err[0] = 0;
    if (!bytes) return fail(AL_EINVAL, "al_apollo_workspace_bytes: bytes is NULL");
    al_status st = check_apollo_cfg(cfg);
    if (st != AL_OK) return st;
    ApolloPlan P;
    if ((st = apollo_plan(tensors, nt, cfg, nullptr, P)) != AL_OK) return st;
    *bytes = P.bytes;
    return AL_OK;
}

al_status al_apollo_step(const al_apollo_tensor* tensors, int32_t nt, const al_apollo_cfg* cfg, int64_t step,
                         void* ws, size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    al_status st = check_apollo_cfg(cfg);
    if (st != AL_OK) return st;
    if (step < 1) return fail(AL_EINVAL, "al_apollo_step: step must be >= 1");
    ApolloPlan P;
    if ((st = apollo_plan(tensors, nt, cfg, nullptr, P)) != AL_OK) return st;
    if (P.desc.empty()) return AL_OK;
    if ((st = check_ws(ws, ws_bytes, P.bytes, "al_apollo_step")) != AL_OK) return st;
    if ((st = apollo_plan(tensors, nt, cfg, static_cast<char*>(ws), P)) != AL_OK) return st;

    al::ApolloArgs a;
    std::memset(&a, 0, sizeof(a));
    a.D = reinterpret_cast<const al::ApolloDesc*>(ws);
    a.nt = (int32_t)P.desc.size();
    a.rank = cfg->rank;
    a.total_tiles = P.total_tiles;
    a.total_chans = P.total_chans;
    a.total_units = P.total_units;
    a.any_whole = P.any_whole;
    a.any_ragged = P.any_ragged;
    a.lr = cfg->lr;
    a.decay = 1.0 - cfg->lr * cfg->weight_decay;
    a.gamma = cfg->gamma;
    a.step = step;

    // the fused AdamW step over the projected moments: gradient R, parameter Rt
    // (cleared by the projection), lr 1, no weight decay -> Rt = -direction;
    // at rank 256 no parameter stream: the step writes the channel scales
    const bool fused = apollo_fused(cfg->rank);
    al::AdamWLaunch w;
    std::memset(&w, 0, sizeof(w));
    const double bc1 = 1.0 - std::pow(cfg->beta1, (double)step);
    const double bc2 = 1.0 - std::pow(cfg->beta2, (double)step);
    w.beta1 = cfg->beta1;
    w.omb1 = 1.0 - cfg->beta1;
    w.beta2 = cfg->beta2;
    w.omb2 = 1.0 - cfg->beta2;
    w.step_size = (float)(1.0 / bc1);
    w.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
    w.eps = (float)cfg->eps;
    w.decay = 1.0f;
    w.v_floor = cfg->v.log_floor;
    w.apollo = fused ? a.D : nullptr;  // descriptor i of the AdamW table is projected tensor i
    const int T = al::adamw_tile_elems(cfg->v.codec, cfg->v.block);
    std::vector<al::AdamWDesc> wd(P.desc.size());
    for (size_t k = 0; k < P.desc.size(); ++k) {
        const al::ApolloDesc& d = P.desc[k];
        const al_apollo_tensor& t = tensors[P.idx[k]];
        al::AdamWDesc& x = wd[k];
        x.p = d.Rt;
        x.g = d.R;
        x.m = t.m;
        x.ms = t.m_meta;
        x.v = t.v;
        x.vm = t.v_meta;
        x.n = d.C * cfg->rank;
        x.tile_begin = w.total_tiles;
        w.total_tiles += (x.n + T - 1) / T;
    }

    hipStream_t s = as_stream(stream);
    hipError_t e;
    if ((e = al::apollo_copy_desc(P.desc.data(), a.nt, const_cast<al::ApolloDesc*>(a.D), s)) != hipSuccess ||
        (e = al::launch_apollo_proj(a, cfg->grad_dtype, s)) != hipSuccess ||
        (e = al::adamw_write_table(wd.data(), (int)wd.size(), static_cast<char*>(ws) + P.adamw_off, w, s)) !=
            hipSuccess ||
        (e = al::launch_adamw(w, AL_DTYPE_F32, cfg->m.codec, cfg->v.codec, cfg->v.block, s, fused)) != hipSuccess)
        return hip_fail(e, "al_apollo_step launch");
    if ((!fused && (e = al::launch_apollo_scale(a, s)) != hipSuccess) ||
        (e = al::launch_apollo_norm(a, s)) != hipSuccess || (e = al::launch_apollo_update(a, cfg->grad_dtype, s)) != hipSuccess)
        return hip_fail(e, "al_apollo_step launch");
    return AL_OK;
}

al_status al_diag_math(int32_t fn, const double* x, int64_t n, double* out, void* stream) {
    g_err[0] = 0;
    if (fn < 0 || fn > 10) return fail(AL_EINVAL, "al_diag_math: fn %d", fn);
    if (n < 0) return fail(AL_EINVAL, "al_diag_math: n < 0");
    if (fn >= 9 && n % 8 != 0) return fail(AL_EINVAL, "al_diag_math: fn 9 and 10 take groups of 8 inputs");
    if (n == 0) return AL_OK;
    if (!x || !out) return fail(AL_EINVAL, "al_diag_math: NULL buffer");
    if (!aligned16(x) || !aligned16(out)) return fail(AL_EALIGN, "al_diag_math: alignment");
    hipError_t e = al::launch_diag_math(fn, x, n, out, al::device_cu_count() * 8, as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_diag_math launch");
}

al_status al_diag_levels(int32_t kind, const float* meta, int64_t nblocks, double* out, void* stream) {
    g_err[0] = 0;
    if (kind < 0 || kind > 1) return fail(AL_EINVAL, "al_diag_levels: kind %d", kind);
    if (nblocks < 0 || nblocks > (int64_t(1) << 40)) return fail(AL_EINVAL, "al_diag_levels: nblocks out of range");
    if (nblocks == 0) return AL_OK;
    if (!meta || !out) return fail(AL_EINVAL, "al_diag_levels: NULL buffer");
    if (!aligned16(meta) || !aligned16(out)) return fail(AL_EALIGN, "al_diag_levels: alignment");
    hipError_t e = al::launch_diag_levels(kind, meta, nblocks, out, al::device_cu_count() * 8, as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_diag_levels launch");
}

al_status al_diff_norms(const float* a, const float* b, int64_t n, double* out, void* stream) {
    g_err[0] = 0;
    if (n < 0) return fail(AL_EINVAL, "al_diff_norms: n < 0");
    if (!out) return fail(AL_EINVAL, "al_diff_norms: out is NULL");
    if (n > 0 && (!a || !b)) return fail(AL_EINVAL, "al_diff_norms: NULL buffer");
    if (!aligned16(out) || (n > 0 && (!aligned16(a) || !aligned16(b))))
        return fail(AL_EALIGN, "al_diff_norms: alignment");
    hipError_t e = al::launch_diff_norms(a, b, n, out, as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_diff_norms launch");
}

al_status al_diag_stream(int32_t mode, float* p, const void* g, void* m, void* v, int64_t n, void* stream) {
    g_err[0] = 0;
    if (mode < 0 || mode > 3) return fail(AL_EINVAL, "al_diag_stream: mode must be 0..3");
    const int64_t unit = (mode & 2) ? 4096 : 2048;
    if (n < 0 || n % unit != 0)
        return fail(AL_EINVAL, "al_diag_stream: n must be a non-negative multiple of 2048 (4096 for the wide shape)");
    if (n == 0) return AL_OK;
    if (!p || !g || !m || !v) return fail(AL_EINVAL, "al_diag_stream: NULL buffer");
    if (!aligned16(p) || !aligned16(g) || !aligned16(m) || !aligned16(v))
        return fail(AL_EALIGN, "al_diag_stream: alignment");
    hipError_t e = al::launch_diag_stream(mode, p, static_cast<const uint16_t*>(g),
                                          static_cast<uint8_t*>(m), static_cast<uint8_t*>(v), n, as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_diag_stream launch");
}

al_status al_synth_normal(void* out, int32_t out_dtype, int64_t n, uint64_t key, float scale, uint64_t mask_key,
                          uint64_t mask_threshold, void* stream) {
    g_err[0] = 0;
    if (out_dtype != AL_DTYPE_F32 && out_dtype != AL_DTYPE_BF16) return fail(AL_EINVAL, "al_synth_normal: dtype");
    if (n < 0) return fail(AL_EINVAL, "al_synth_normal: n < 0");
    if (n == 0) return AL_OK;
    if (!out) return fail(AL_EINVAL, "al_synth_normal: out is NULL");
    if (!aligned16(out)) return fail(AL_EALIGN, "al_synth_normal: alignment");
    hipError_t e = al::launch_synth_normal(out, out_dtype == AL_DTYPE_BF16, n, key, scale, mask_key, mask_threshold,
                                           al::device_cu_count() * 16, as_stream(stream));
    return e == hipSuccess ? AL_OK : hip_fail(e, "al_synth_normal launch");
}

al_status al_adafactor_workspace_bytes(const al_tensor* tensors, int32_t nt, const al_adafactor_cfg* cfg,
                                       size_t* bytes) {
    g_err[0] = 0;
    if (!bytes) return fail(AL_EINVAL, "al_adafactor_workspace_bytes: bytes is NULL");
    *bytes = 0;
    al_status st = check_adafactor_cfg(cfg);
    if (st != AL_OK) return st;
    FacPlan P;
    if ((st = fac_plan(tensors, nt, false, kNoSpec, cfg->v, kNoSpec, nullptr, P)) != AL_OK) return st;
    *bytes = P.bytes;
    return AL_OK;
}

al_status al_came_workspace_bytes(const al_tensor* tensors, int32_t nt, const al_came_cfg* cfg, size_t* bytes) {
    g_err[0] = 0;
    if (!bytes) return fail(AL_EINVAL, "al_came_workspace_bytes: bytes is NULL");
    *bytes = 0;
    al_status st = check_came_cfg(cfg);
    if (st != AL_OK) return st;
    FacPlan P;
    if ((st = fac_plan(tensors, nt, true, cfg->m, cfg->v, cfg->conf, nullptr, P)) != AL_OK) return st;
    *bytes = P.bytes;
    return AL_OK;
}

al_status al_adafactor_step(const al_tensor* tensors, int32_t nt, const al_adafactor_cfg* cfg, int64_t step,
                            void* ws, size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    al_status st = check_adafactor_cfg(cfg);
    if (st != AL_OK) return st;
    if (step < 1) return fail(AL_EINVAL, "al_adafactor_step: step must be >= 1");
    FacPlan P;
    if ((st = fac_plan(tensors, nt, false, kNoSpec, cfg->v, kNoSpec, nullptr, P)) != AL_OK) return st;
    if (P.desc.empty()) return AL_OK;
    if ((st = check_ws(ws, ws_bytes, P.bytes, "al_adafactor_step")) != AL_OK) return st;
    if ((st = fac_plan(tensors, nt, false, kNoSpec, cfg->v, kNoSpec, static_cast<char*>(ws), P)) != AL_OK) return st;

    al::FacArgs a = fac_args(P, static_cast<char*>(ws));
    a.beta = 1.0 - std::pow((double)step, cfg->decay_rate);
    a.omb = 1.0 - a.beta;
    a.eps1 = cfg->eps1;
    a.lr = cfg->lr;
    a.decay = 1.0 - cfg->lr * cfg->weight_decay;
    a.clip_d = cfg->clip_threshold;
    a.v_codec = cfg->v.codec;
    a.v_block = cfg->v.block;
    a.v_floor = cfg->v.log_floor;
    a.exact_all = (cfg->flags & AL_FLAG_EXACT_SUMS) != 0;
    hipStream_t s = as_stream(stream);
    const int G = cfg->grad_dtype;
    hipError_t e;
    if ((e = al::fac_copy_desc(P.desc.data(), (int)P.desc.size(), const_cast<al::FacDesc*>(a.D), s)) != hipSuccess ||
        (e = al::launch_fac_marg_g2(a, G, s)) != hipSuccess || (e = al::launch_fac_fin(a, 0, G, s)) != hipSuccess ||
        (e = al::launch_fac_rms(a, G, s)) != hipSuccess || (e = al::launch_fac_clip(a, s)) != hipSuccess ||
        (e = al::launch_ada_apply(a, G, s)) != hipSuccess || (e = al::launch_ada_vec1d(a, G, s)) != hipSuccess)
        return hip_fail(e, "al_adafactor_step launch");
    return AL_OK;
}

al_status al_came_step(const al_tensor* tensors, int32_t nt, const al_came_cfg* cfg, int64_t step, void* ws,
                       size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    al_status st = check_came_cfg(cfg);
    if (st != AL_OK) return st;
    if (step < 1) return fail(AL_EINVAL, "al_came_step: step must be >= 1");
    FacPlan P;
    if ((st = fac_plan(tensors, nt, true, cfg->m, cfg->v, cfg->conf, nullptr, P)) != AL_OK) return st;
    if (P.desc.empty()) return AL_OK;
    if ((st = check_ws(ws, ws_bytes, P.bytes, "al_came_step")) != AL_OK) return st;
    if ((st = fac_plan(tensors, nt, true, cfg->m, cfg->v, cfg->conf, static_cast<char*>(ws), P)) != AL_OK) return st;

    al::FacArgs a = fac_args(P, static_cast<char*>(ws));
    a.beta = cfg->beta2;
    a.omb = 1.0 - cfg->beta2;
    a.beta1 = cfg->beta1;
    a.omb1 = 1.0 - cfg->beta1;
    a.beta3 = cfg->beta3;
    a.omb3 = 1.0 - cfg->beta3;
    a.eps1 = cfg->eps1;
    a.eps2 = cfg->eps2;
    a.lr = cfg->lr;
    a.decay = 1.0 - cfg->lr * cfg->weight_decay;
    a.clip_d = cfg->clip_threshold;
    a.v_codec = cfg->v.codec;
    a.v_block = cfg->v.block;
    a.v_floor = cfg->v.log_floor;
    a.c_codec = cfg->conf.codec;
    a.c_block = cfg->conf.block;
    a.c_floor = cfg->conf.log_floor;
    a.m_codec = cfg->m.codec;
    a.m_block = cfg->m.codec == AL_CODEC_UF8 ? cfg->m.block : 256;
    a.exact_all = (cfg->flags & AL_FLAG_EXACT_SUMS) != 0;
    hipStream_t s = as_stream(stream);
    const int G = cfg->grad_dtype;
    hipError_t e;
    if ((e = al::fac_copy_desc(P.desc.data(), (int)P.desc.size(), const_cast<al::FacDesc*>(a.D), s)) != hipSuccess ||
        (e = al::launch_fac_marg_g2(a, G, s)) != hipSuccess || (e = al::launch_fac_fin(a, 0, G, s)) != hipSuccess ||
        (e = al::launch_fac_rms(a, G, s)) != hipSuccess || (e = al::launch_fac_clip(a, s)) != hipSuccess ||
        (e = al::launch_came_res(a, G, s)) != hipSuccess || (e = al::launch_fac_fin(a, 1, G, s)) != hipSuccess ||
        (e = al::launch_came_apply(a, G, s)) != hipSuccess || (e = al::launch_came_vec1d(a, G, s)) != hipSuccess)
        return hip_fail(e, "al_came_step launch");
    return AL_OK;
}

}  // extern "C"
