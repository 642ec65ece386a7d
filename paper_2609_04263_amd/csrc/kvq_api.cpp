// Host side of the C ABI declared in include/kvq.h: format validation, the
// storage layout, argument checks (all before any launch, so an error
// changes nothing) and kernel dispatch on the caller's stream.

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "kvq_internal.h"

namespace {

bool pow2_in(int v, int lo, int hi)
{
    return v >= lo && v <= hi && (v & (v - 1)) == 0;
}

kvq_status check_format(const kvq_format* f, int D)
{
    if (!f)
        return KVQ_ERR_ARG;
    if (D != 64 && D != 128 && D != 256)
        return KVQ_ERR_FORMAT;
    if ((f->k_bits != 2 && f->k_bits != 4 && f->k_bits != 8) || (f->v_bits != 2 && f->v_bits != 4 && f->v_bits != 8))
        return KVQ_ERR_FORMAT;
    if ((f->k_bits == 8) != (f->v_bits == 8))  // 8-bit codes: keys and values both
        return KVQ_ERR_FORMAT;
    if ((f->k_mode != KVQ_AFFINE && f->k_mode != KVQ_SYMMETRIC) ||
        (f->v_mode != KVQ_AFFINE && f->v_mode != KVQ_SYMMETRIC))
        return KVQ_ERR_FORMAT;
    if ((f->k_axis != KVQ_PER_TOKEN && f->k_axis != KVQ_PER_CHANNEL) || f->v_axis != KVQ_PER_TOKEN)
        return KVQ_ERR_FORMAT;
    if (f->residual < 0 || f->flush < 0 || (f->flush == 0 && f->residual != 0) || f->flush % 32 != 0)
        return KVQ_ERR_FORMAT;
    if (f->rotate != 0 && f->rotate != D)
        return KVQ_ERR_FORMAT;
    if (f->k_axis == KVQ_PER_TOKEN ? !pow2_in(f->k_group, 32, D) : (f->k_group != 32 || f->flush == 0))
        return KVQ_ERR_FORMAT;
    if (!pow2_in(f->v_group, 32, D))
        return KVQ_ERR_FORMAT;
    if (f->meta_fp16 != 0 && f->meta_fp16 != 1)
        return KVQ_ERR_FORMAT;
    if (f->sink < 0 || f->sink % 32 != 0)
        return KVQ_ERR_FORMAT;
    return KVQ_OK;
}

size_t round_up(size_t v, size_t a)
{
    return (v + a - 1) / a * a;
}

// Tail capacity per (b, h): T_max - sink rounded up to 32 (0 when the sink
// covers T_max).
size_t tail_alloc(const kvq_format& f, int T_max)
{
    return T_max > f.sink ? round_up((size_t)(T_max - f.sink), 32) : 0;
}

kvq_status layout(const kvq_format* f, int B, int H, int D, int T_max, size_t off[10], size_t len[10], size_t* total)
{
    kvq_status st = check_format(f, D);
    if (st != KVQ_OK)
        return st;
    if (B < 1 || H < 1 || T_max < 1)
        return KVQ_ERR_ARG;
    const size_t bh = (size_t)B * H, T = tail_alloc(*f, T_max);
    const size_t ring = (size_t)(f->residual + f->flush);
    len[0] = bh * T * (size_t)(D * f->k_bits / 32) * 4;
    const size_t msz = f->meta_fp16 ? 2 : 4;  // bytes per scale or offset
    len[1] = f->k_axis == KVQ_PER_TOKEN ? bh * T * (size_t)(D / f->k_group) * msz : bh * (T / 32) * (size_t)D * msz;
    len[2] = f->k_mode == KVQ_AFFINE ? len[1] : 0;
    len[3] = bh * (T * f->v_bits / 32) * (size_t)D * 4;
    len[4] = bh * T * (size_t)(D / f->v_group) * msz;
    len[5] = f->v_mode == KVQ_AFFINE ? len[4] : 0;
    len[6] = f->flush ? bh * ring * (size_t)D * 2 : 0;
    len[7] = len[6];
    len[8] = bh * (size_t)f->sink * (size_t)D * 2;
    len[9] = len[8];
    size_t o = 0;
    for (int i = 0; i < 10; ++i) {
        off[i] = o;
        o = round_up(o + len[i], 256);
    }
    *total = o;
    return KVQ_OK;
}

bool aligned16(const void* p)
{
    return ((uintptr_t)p & 15u) == 0;
}

bool same_format(const kvq_format& a, const kvq_format& b)
{
    return memcmp(&a, &b, sizeof(kvq_format)) == 0;
}

float rotation_constant(int D)
{
    return (float)(1.0 / sqrt((double)D));  // binary32 value nearest D^(-1/2)
}

// Decode workspace: partial outputs fp32 [B*H_q][S][D], then partial
// (max, sum) fp32 [B*H_q][S][2], sized for the largest split count S the
// cache can need (the split count of a call never exceeds it).
size_t decode_workspace_layout(const kvq_cache* c, int H_q, size_t* off_ml)
{
    int S_max = kvq::decode_split_bound(c->B, c->H);
    size_t rows = (size_t)c->B * H_q;
    size_t o_ml = round_up(rows * S_max * c->D * sizeof(float), 256);
    if (off_ml)
        *off_ml = o_ml;
    return o_ml + rows * S_max * 2 * sizeof(float);
}

template <typename T>
T* at(const kvq_cache* c, int section)
{
    return (T*)(c->base + c->off[section]);
}

}  // namespace

namespace kvq {

LaunchTiming& launch_timing()
{
    static thread_local LaunchTiming t;
    return t;
}

int num_tail(const kvq_format& f, int n)
{
    return n > f.sink ? n - f.sink : 0;
}

int num_coded(const kvq_format& f, int n)
{
    n = num_tail(f, n);
    if (f.flush == 0)
        return n;
    int over = n - f.residual;
    return over <= 0 ? 0 : over / f.flush * f.flush;
}

}  // namespace kvq

namespace {

// One decode step of a window format through the projection: row b of H is
// sequence b's new token (M = B).  The stream kernel writes Q, and K and V
// straight into the token's fp16 window slot; a flush that falls due (the
// oldest tokens of a full window leaving it) is then coded from the window
// by the block coder, exactly as kvq_append of the same bf16 K and V does.
// The new token is never among the flushed ones (the window keeps at least
// `residual` >= 1 tokens), so the coder reads only window rows.
kvq_status project_append_window(const void* H, int M, int d_in, const void* W, int d_q, int d_kv, const void* A,
                                 const void* Bm, int rank, float lora_scale, void* Q, kvq_cache* c, void* workspace,
                                 size_t ws_bytes, void* stream)
{
    const kvq_format& f = c->fmt;
    if (f.rotate != 0 || f.sink != 0 || f.residual < 1)
        return KVQ_ERR_FORMAT;
    if (M != c->B || M > 32 || d_in < 64 || d_in % 64 != 0 || d_q < 16 || d_q % 16 != 0 || d_kv != c->H * c->D)
        return KVQ_ERR_ARG;
    if (rank < 0 || rank > 64 || !isfinite(lora_scale))
        return KVQ_ERR_ARG;
    if (!H || !W || !Q || !aligned16(H) || !aligned16(W) || !aligned16(Q))
        return KVQ_ERR_ARG;
    if (rank > 0) {
        if (!A || !Bm || !aligned16(A) || !aligned16(Bm) || !workspace || !aligned16(workspace))
            return KVQ_ERR_ARG;
        if (ws_bytes < kvq::project_workspace_bytes(M, rank))
            return KVQ_ERR_WORKSPACE;
    }
    if ((long long)c->n + 1 > c->T_max)
        return KVQ_ERR_CAPACITY;
    hipStream_t s = (hipStream_t)stream;
    const int n0 = c->n, n1 = n0 + 1, ring = f.residual + f.flush;
    kvq::ProjParams p = {};
    p.x = (const uint16_t*)H;
    p.w = (const uint16_t*)W;
    p.a = (const uint16_t*)A;
    p.bm = (const uint16_t*)Bm;
    p.t = (const float*)workspace;
    p.y0 = (uint16_t*)Q;
    p.M = M;
    p.K = d_in;
    p.N = d_q + 2 * d_kv;
    p.n1 = d_q;
    p.n2 = d_q + d_kv;
    p.rank = rank;
    p.scale = lora_scale;
    p.kr = at<uint16_t>(c, 6);
    p.vr = at<uint16_t>(c, 7);
    p.rslots = ring;
    p.rslot = n0 % ring;
    p.cH = c->H;
    p.cD = c->D;
    if (kvq::launch_project_decode(p, s) != hipSuccess)
        return KVQ_ERR_DEVICE;
    const int q0 = kvq::num_coded(f, n0), q1 = kvq::num_coded(f, n1);
    if (q1 > q0) {
        kvq::AppendParams a = {};
        a.kc = at<uint32_t>(c, 0);
        a.ks = at<float>(c, 1);
        a.kz = at<float>(c, 2);
        a.vc = at<uint32_t>(c, 3);
        a.vs = at<float>(c, 4);
        a.vz = at<float>(c, 5);
        a.kr = p.kr;
        a.vr = p.vr;
        a.kin = p.kr;  // never read: every flushed token is in the window
        a.vin = p.vr;
        a.B = c->B;
        a.H = c->H;
        a.T = c->T_alloc;
        a.n_new = 1;
        a.k_bits = f.k_bits;
        a.v_bits = f.v_bits;
        a.k_mode = f.k_mode;
        a.v_mode = f.v_mode;
        a.k_axis = f.k_axis;
        a.k_group = f.k_group;
        a.v_group = f.v_group;
        a.rotate = 0;
        a.rot_c = rotation_constant(c->D);
        a.meta16 = f.meta_fp16;
        a.n0 = n0;
        a.q0 = q0;
        a.q1 = q1;
        a.ring = ring;
        a.ring_lo = n1;  // the new row is already in its slot
        if (kvq::launch_append(a, c->D, s) != hipSuccess)
            return KVQ_ERR_DEVICE;
    }
    c->n = n1;
    return KVQ_OK;
}

}  // namespace

extern "C" {

kvq_status kvq_time_launches(void* start_event, void* stop_event)
{
    if ((start_event == nullptr) != (stop_event == nullptr))
        return KVQ_ERR_ARG;
    kvq::LaunchTiming& t = kvq::launch_timing();
    t.start = (hipEvent_t)start_event;
    t.stop = (hipEvent_t)stop_event;
    return KVQ_OK;
}

const char* kvq_strerror(kvq_status s)
{
    switch (s) {
    case KVQ_OK:
        return "ok";
    case KVQ_ERR_ARG:
        return "invalid argument";
    case KVQ_ERR_FORMAT:
        return "unsupported or mismatched cache format";
    case KVQ_ERR_CAPACITY:
        return "cache capacity exceeded";
    case KVQ_ERR_WORKSPACE:
        return "workspace too small";
    case KVQ_ERR_DEVICE:
        return "HIP device error";
    case KVQ_ERR_SCRATCH:
        return "call needs more split-partial memory than the static scratch (KVQ_SCRATCH_BYTES)";
    }
    return "unknown status";
}

kvq_status kvq_cache_bytes(const kvq_format* fmt, int B, int H_kv, int D, int T_max, size_t* bytes)
{
    if (!bytes)
        return KVQ_ERR_ARG;
    size_t off[10], len[10];
    return layout(fmt, B, H_kv, D, T_max, off, len, bytes);
}

kvq_status kvq_cache_init(const kvq_format* fmt, int B, int H_kv, int D, int T_max, void* storage, size_t bytes,
                          kvq_cache** out)
{
    if (!out || !storage || ((uintptr_t)storage & 255u))
        return KVQ_ERR_ARG;
    size_t off[10], len[10], total;
    kvq_status st = layout(fmt, B, H_kv, D, T_max, off, len, &total);
    if (st != KVQ_OK)
        return st;
    if (bytes < total)
        return KVQ_ERR_ARG;
    kvq_cache* c = (kvq_cache*)calloc(1, sizeof(kvq_cache));
    if (!c)
        return KVQ_ERR_ARG;
    c->fmt = *fmt;
    c->B = B;
    c->H = H_kv;
    c->D = D;
    c->T_max = T_max;
    c->T_alloc = (int)tail_alloc(*fmt, T_max);
    c->base = (uint8_t*)storage;
    c->bytes = bytes;
    memcpy(c->off, off, sizeof(off));
    memcpy(c->len, len, sizeof(len));
    c->n = 0;
    *out = c;
    return KVQ_OK;
}

kvq_status kvq_cache_section(const kvq_cache* c, int index, size_t* offset, size_t* length)
{
    if (!c || index < 0 || index > 9 || !offset || !length)
        return KVQ_ERR_ARG;
    *offset = c->off[index];
    *length = c->len[index];
    return KVQ_OK;
}

kvq_status kvq_cache_reset(kvq_cache* c)
{
    if (!c)
        return KVQ_ERR_ARG;
    c->n = 0;
    return KVQ_OK;
}

kvq_status kvq_cache_len(const kvq_cache* c, int* n, int* n_coded)
{
    if (!c || !n || !n_coded)
        return KVQ_ERR_ARG;
    *n = c->n;
    *n_coded = kvq::num_coded(c->fmt, c->n);
    return KVQ_OK;
}

kvq_status kvq_cache_rewind(kvq_cache* c, int n_new)
{
    if (!c || n_new < 0 || n_new > c->n)
        return KVQ_ERR_ARG;
    if (c->fmt.flush != 0)
        return KVQ_ERR_FORMAT;
    c->n = n_new;
    return KVQ_OK;
}

kvq_status kvq_cache_restore(kvq_cache* c, int n)
{
    if (!c || n < 0 || n > c->T_max)
        return KVQ_ERR_ARG;
    c->n = n;
    return KVQ_OK;
}

void kvq_cache_destroy(kvq_cache* c)
{
    free(c);
}

kvq_status kvq_project_workspace_bytes(int M, int rank, size_t* bytes)
{
    if (!bytes || M < 0 || rank < 0 || rank > 64)
        return KVQ_ERR_ARG;
    *bytes = kvq::project_workspace_bytes(M, rank);
    return KVQ_OK;
}

kvq_status kvq_project_qkv(const void* H, int M, int d_in, const void* W, int d_q, int d_kv, const void* A,
                           const void* Bm, int rank, float lora_scale, void* Q, void* K, void* V, void* workspace,
                           size_t ws_bytes, void* stream)
{
    if (M < 0 || d_in < 64 || d_in % 64 != 0 || d_q < 16 || d_kv < 16 || d_q % 16 != 0 || d_kv % 16 != 0)
        return KVQ_ERR_ARG;
    if (rank < 0 || rank > 64 || !isfinite(lora_scale))
        return KVQ_ERR_ARG;
    if (M == 0)
        return KVQ_OK;
    if (!H || !W || !Q || !K || !V || !aligned16(H) || !aligned16(W) || !aligned16(Q) || !aligned16(K) ||
        !aligned16(V))
        return KVQ_ERR_ARG;
    if (rank > 0) {
        if (!A || !Bm || !aligned16(A) || !aligned16(Bm) || !workspace || !aligned16(workspace))
            return KVQ_ERR_ARG;
        if (ws_bytes < kvq::project_workspace_bytes(M, rank))
            return KVQ_ERR_WORKSPACE;
    }
    hipStream_t s = (hipStream_t)stream;
    const int N = d_q + 2 * d_kv;
    if (M <= 32) {
        // decode: partial adapter activations over K slices, then the weight stream
        kvq::ProjParams p = {};
        p.x = (const uint16_t*)H;
        p.w = (const uint16_t*)W;
        p.a = (const uint16_t*)A;
        p.bm = (const uint16_t*)Bm;
        p.t = (const float*)workspace;
        p.y0 = (uint16_t*)Q;
        p.y1 = (uint16_t*)K;
        p.y2 = (uint16_t*)V;
        p.M = M;
        p.K = d_in;
        p.N = N;
        p.n1 = d_q;
        p.n2 = d_q + d_kv;
        p.rank = rank;
        p.scale = lora_scale;
        return kvq::launch_project(p, s) == hipSuccess ? KVQ_OK : KVQ_ERR_DEVICE;
    }
    // large-M pass: with the adapter streamed as extra K stages the
    // activation pass writes bf16 hi / lo activations instead of fp32
    const bool hilo = kvq::project_adapter_stages(M, d_in, d_q, d_kv, rank);
    if (rank > 0) {
        kvq::ProjParams a = {};
        a.x = (const uint16_t*)H;
        a.w = (const uint16_t*)A;
        a.yf = (float*)workspace;
        a.t_hilo = hilo;
        a.M = M;
        a.K = d_in;
        a.N = 3 * rank;
        a.n1 = a.n2 = 3 * rank;
        a.rank = 0;
        a.scale = lora_scale;
        if (kvq::launch_project(a, s) != hipSuccess)
            return KVQ_ERR_DEVICE;
    }
    kvq::ProjParams p = {};
    p.x = (const uint16_t*)H;
    p.w = (const uint16_t*)W;
    p.bm = (const uint16_t*)Bm;
    p.t = (const float*)workspace;
    p.y0 = (uint16_t*)Q;
    p.y1 = (uint16_t*)K;
    p.y2 = (uint16_t*)V;
    p.M = M;
    p.K = d_in;
    p.N = N;
    p.n1 = d_q;
    p.n2 = d_q + d_kv;
    p.rank = rank;
    p.scale = 1.0f;
    p.t_hilo = hilo;
    return kvq::launch_project(p, s) == hipSuccess ? KVQ_OK : KVQ_ERR_DEVICE;
}

kvq_status kvq_project_append(const void* H, int M, int d_in, const void* W, int d_q, int d_kv, const void* A,
                              const void* Bm, int rank, float lora_scale, void* Q, kvq_cache* c, int n_new,
                              void* workspace, size_t ws_bytes, void* stream)
{
    if (!c || n_new < 0)
        return KVQ_ERR_ARG;
    const kvq_format& f = c->fmt;
    if (n_new == 1 && f.flush > 0)
        return project_append_window(H, M, d_in, W, d_q, d_kv, A, Bm, rank, lora_scale, Q, c, workspace, ws_bytes,
                                     stream);
    if (f.k_axis != KVQ_PER_TOKEN || f.flush != 0 || f.rotate != 0 || f.sink != 0)
        return KVQ_ERR_FORMAT;
    if (M < 256 || d_in < 64 || d_in % 64 != 0 || d_q % 256 != 0 || d_kv % 256 != 0 || d_kv != c->H * c->D)
        return KVQ_ERR_ARG;
    if (n_new % 32 != 0 || c->n % 32 != 0 || (long long)c->B * n_new != M)
        return KVQ_ERR_ARG;
    if (rank < 0 || rank > 64 || !isfinite(lora_scale))
        return KVQ_ERR_ARG;
    if (!H || !W || !Q || !aligned16(H) || !aligned16(W) || !aligned16(Q))
        return KVQ_ERR_ARG;
    if (rank > 0) {
        if (!A || !Bm || !aligned16(A) || !aligned16(Bm) || !workspace || !aligned16(workspace))
            return KVQ_ERR_ARG;
        if (ws_bytes < kvq::project_workspace_bytes(M, rank))
            return KVQ_ERR_WORKSPACE;
    }
    if ((long long)c->n + n_new > c->T_max)
        return KVQ_ERR_CAPACITY;
    hipStream_t s = (hipStream_t)stream;
    if (rank > 0) {
        kvq::ProjParams a = {};
        a.x = (const uint16_t*)H;
        a.w = (const uint16_t*)A;
        a.yf = (float*)workspace;
        a.M = M;
        a.K = d_in;
        a.N = 3 * rank;
        a.n1 = a.n2 = 3 * rank;
        a.rank = 0;
        a.scale = lora_scale;
        if (kvq::launch_project(a, s) != hipSuccess)
            return KVQ_ERR_DEVICE;
    }
    kvq::ProjParams p = {};
    p.x = (const uint16_t*)H;
    p.w = (const uint16_t*)W;
    p.bm = (const uint16_t*)Bm;
    p.t = (const float*)workspace;
    p.y0 = (uint16_t*)Q;
    p.M = M;
    p.K = d_in;
    p.N = d_q + 2 * d_kv;
    p.n1 = d_q;
    p.n2 = d_q + d_kv;
    p.rank = rank;
    p.scale = 1.0f;
    p.fuse = 1;
    p.kc = at<uint32_t>(c, 0);
    p.ks = at<float>(c, 1);
    p.kz = at<float>(c, 2);
    p.vc = at<uint32_t>(c, 3);
    p.vs = at<float>(c, 4);
    p.vz = at<float>(c, 5);
    p.cH = c->H;
    p.cD = c->D;
    p.cT = c->T_alloc;
    p.cn0 = c->n;
    p.cn_new = n_new;
    p.k_bits = f.k_bits;
    p.v_bits = f.v_bits;
    p.k_mode = f.k_mode;
    p.v_mode = f.v_mode;
    p.k_group = f.k_group;
    p.v_group = f.v_group;
    p.meta16 = f.meta_fp16;
    if (kvq::launch_project(p, s) != hipSuccess)
        return KVQ_ERR_DEVICE;
    c->n += n_new;
    return KVQ_OK;
}

kvq_status kvq_merge_adapter(const void* W, int d_in, int d_q, int d_kv, const void* A, const void* Bm, int rank,
                             float lora_scale, void* Wout, void* stream)
{
    if (d_in < 64 || d_in % 64 != 0 || d_q < 32 || d_kv < 32 || d_q % 32 != 0 || d_kv % 32 != 0)
        return KVQ_ERR_ARG;
    if (rank < 1 || rank > 64 || !isfinite(lora_scale))
        return KVQ_ERR_ARG;
    if (!W || !A || !Bm || !Wout || !aligned16(W) || !aligned16(A) || !aligned16(Bm) || !aligned16(Wout))
        return KVQ_ERR_ARG;
    kvq::MergeParams p = {};
    p.w = (const uint16_t*)W;
    p.a = (const uint16_t*)A;
    p.bm = (const uint16_t*)Bm;
    p.out = (uint16_t*)Wout;
    p.d_in = d_in;
    p.d_q = d_q;
    p.d_kv = d_kv;
    p.rank = rank;
    p.scale = lora_scale;
    return kvq::launch_merge(p, (hipStream_t)stream) == hipSuccess ? KVQ_OK : KVQ_ERR_DEVICE;
}

kvq_status kvq_append(kvq_cache* c, const void* K, const void* V, int n_new, const kvq_format* fmt, void* stream)
{
    if (!c || !fmt || n_new < 0)
        return KVQ_ERR_ARG;
    if (!same_format(c->fmt, *fmt))
        return KVQ_ERR_FORMAT;
    if (n_new == 0)
        return KVQ_OK;
    if (!K || !V || !aligned16(K) || !aligned16(V))
        return KVQ_ERR_ARG;
    if ((long long)c->n + n_new > c->T_max)
        return KVQ_ERR_CAPACITY;
    const kvq_format& f = c->fmt;
    kvq::AppendParams p = {};
    p.kc = at<uint32_t>(c, 0);
    p.ks = at<float>(c, 1);
    p.kz = at<float>(c, 2);
    p.vc = at<uint32_t>(c, 3);
    p.vs = at<float>(c, 4);
    p.vz = at<float>(c, 5);
    p.kr = at<uint16_t>(c, 6);
    p.vr = at<uint16_t>(c, 7);
    p.kin = (const uint16_t*)K;
    p.vin = (const uint16_t*)V;
    p.B = c->B;
    p.H = c->H;
    p.T = c->T_alloc;
    p.n_new = n_new;
    p.k_bits = f.k_bits;
    p.v_bits = f.v_bits;
    p.k_mode = f.k_mode;
    p.v_mode = f.v_mode;
    p.k_axis = f.k_axis;
    p.k_group = f.k_group;
    p.v_group = f.v_group;
    p.rotate = f.rotate;
    p.rot_c = rotation_constant(c->D);
    p.meta16 = f.meta_fp16;
    const int n0 = c->n, n1 = n0 + n_new, S = f.sink;
    if (n0 < S) {
        // sink tokens [n0, min(S, n1)): fp16 rows t of sections 8 and 9
        kvq::AppendParams ps = p;
        ps.kr = at<uint16_t>(c, 8);
        ps.vr = at<uint16_t>(c, 9);
        ps.n0 = n0;
        ps.ring = S;
        ps.ring_lo = n0;
        if (kvq::launch_append_rows(ps, c->D, n1 < S ? n1 : S, (hipStream_t)stream) != hipSuccess)
            return KVQ_ERR_DEVICE;
    }
    if (n1 > S) {
        // the tail, in tail indices; n0 - S < 0 when the call starts in the sink
        p.n0 = n0 - S;
        p.q0 = kvq::num_coded(f, n0);
        p.q1 = kvq::num_coded(f, n1);
        p.ring = f.residual + f.flush;
        const int t0 = n0 > S ? n0 - S : 0, t1 = n1 - S;
        p.ring_lo = p.ring ? (t1 - p.ring > t0 ? t1 - p.ring : t0) : t1;
        if (kvq::launch_append(p, c->D, (hipStream_t)stream) != hipSuccess)
            return KVQ_ERR_DEVICE;
    }
    c->n = n1;
    return KVQ_OK;
}

kvq_status kvq_decode_workspace_bytes(const kvq_cache* c, int H_q, size_t* bytes)
{
    if (!c || !bytes || H_q < c->H || H_q % c->H != 0 || H_q / c->H > 16)
        return KVQ_ERR_ARG;
    // Splits never exceed the bound at the largest coded-token count.
    *bytes = decode_workspace_layout(c, H_q, nullptr);
    return KVQ_OK;
}

}  // extern "C"

namespace {

// Everything of a decode-attention call except its partial-result buffers
// and split plan: argument checks, then the cache sections, dimensions and
// format of the kernel parameters.
kvq_status decode_setup(const kvq_cache* c, const void* Q, int H_q, float sm_scale, void* O, kvq::AttnParams* pp)
{
    if (!c || !Q || !O || !aligned16(Q) || !aligned16(O))
        return KVQ_ERR_ARG;
    if (H_q < c->H || H_q % c->H != 0 || H_q / c->H > 16 || !isfinite(sm_scale))
        return KVQ_ERR_ARG;
    if (c->n < 1)
        return KVQ_ERR_ARG;
    const kvq_format& f = c->fmt;
    kvq::AttnParams& p = *pp;
    p = kvq::AttnParams{};
    p.nq = kvq::num_coded(f, c->n);
    p.kc = at<uint32_t>(c, 0);
    p.ks = at<float>(c, 1);
    p.kz = at<float>(c, 2);
    p.vc = at<uint32_t>(c, 3);
    p.vs = at<float>(c, 4);
    p.vz = at<float>(c, 5);
    p.kr = at<uint16_t>(c, 6);
    p.vr = at<uint16_t>(c, 7);
    p.kq = at<uint16_t>(c, 8);
    p.vq = at<uint16_t>(c, 9);
    p.q = (const uint16_t*)Q;
    p.out = (float*)O;
    p.B = c->B;
    p.H = c->H;
    p.H_q = H_q;
    p.G = H_q / c->H;
    p.T = c->T_alloc;
    p.n = kvq::num_tail(f, c->n);
    p.ring = f.residual + f.flush;
    p.sink = f.sink;
    p.n_sink = c->n < f.sink ? c->n : f.sink;
    p.k_bits = f.k_bits;
    p.v_bits = f.v_bits;
    p.k_mode = f.k_mode;
    p.v_mode = f.v_mode;
    p.k_axis = f.k_axis;
    p.k_group = f.k_group;
    p.v_group = f.v_group;
    p.rotate = f.rotate;
    p.sm_log2 = sm_scale * 1.4426950408889634f;
    p.rot_c = rotation_constant(c->D);
    p.meta16 = f.meta_fp16;
    p.lds_bytes = kvq::decode_lds_bytes(c->D, f, p.G);
    return KVQ_OK;
}

// Target workgroups of the split kernel for this call: one resident round.
int decode_groups(const kvq_cache* c, const kvq::AttnParams& p)
{
    return kvq::decode_target_groups(p, c->D);
}

void decode_finish_plan(const kvq_cache* c, int groups, kvq::AttnParams* p)
{
    kvq::decode_plan(c->B, c->H, kvq::decode_waves(c->D, c->fmt), groups, p->nq, &p->S_q, &p->bps);
    p->S_tot = p->S_q;
}

// ------------------------------------------------ static decode scratch
// Split partials of kvq_decode_attn_noalloc live in this array: one copy per
// GPU, held until the process ends.  Host code never passes the array's name
// to a kernel (on the host it is only a stand-in for the symbol); it uses the
// device address hipGetSymbolAddress returns, looked up once per device with
// that device current.
static __device__ __align__(256) uint8_t scratch[KVQ_SCRATCH_BYTES];

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices];

// Device address of `scratch` on the current device, or null on error.
void* scratch_address()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices)
        return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

kvq_status kvq_decode_attn(const kvq_cache* c, const void* Q, int H_q, float sm_scale, void* O, void* workspace,
                           size_t ws_bytes, void* stream)
{
    if (!workspace || !aligned16(workspace))
        return KVQ_ERR_ARG;
    kvq::AttnParams p;
    const kvq_status st = decode_setup(c, Q, H_q, sm_scale, O, &p);
    if (st != KVQ_OK)
        return st;
    size_t off_ml;
    const size_t need = decode_workspace_layout(c, H_q, &off_ml);
    if (ws_bytes < need)
        return KVQ_ERR_WORKSPACE;
    p.part_o = (float*)workspace;
    p.part_ml = (float*)((uint8_t*)workspace + off_ml);
    decode_finish_plan(c, decode_groups(c, p), &p);
    return kvq::launch_decode(p, c->D, (hipStream_t)stream) == hipSuccess ? KVQ_OK : KVQ_ERR_DEVICE;
}

kvq_status kvq_decode_attn_noalloc(const kvq_cache* c, const void* Q, int H_q, float sm_scale, void* O, void* stream)
{
    kvq::AttnParams p;
    const kvq_status st = decode_setup(c, Q, H_q, sm_scale, O, &p);
    if (st != KVQ_OK)
        return st;
    // The plan of kvq_decode_attn, with the split count capped so that the
    // partials (D + 2 floats per row and split, the (max, sum) pairs
    // starting at a 256-byte boundary) fit the scratch; a single split
    // writes the outputs itself and needs none.
    const size_t rows = (size_t)c->B * H_q;
    const size_t per_split = rows * ((size_t)c->D + 2) * sizeof(float);
    const long cap = (long)((KVQ_SCRATCH_BYTES - 256) / per_split);
    int groups = decode_groups(c, p);
    const int units = c->B * c->H;
    if (cap < 2)
        groups = units;
    else if ((long)groups > cap * units)
        groups = (int)(cap * units);
    decode_finish_plan(c, groups, &p);
    if (p.S_tot > 1) {
        uint8_t* base = (uint8_t*)scratch_address();
        if (!base)
            return KVQ_ERR_DEVICE;
        const size_t off_ml = round_up(rows * p.S_tot * c->D * sizeof(float), 256);
        if (off_ml + rows * p.S_tot * 2 * sizeof(float) > KVQ_SCRATCH_BYTES)
            return KVQ_ERR_SCRATCH;  // not reached: the cap above keeps the plan inside
        p.part_o = (float*)base;
        p.part_ml = (float*)(base + off_ml);
    }
    return kvq::launch_decode(p, c->D, (hipStream_t)stream) == hipSuccess ? KVQ_OK : KVQ_ERR_DEVICE;
}

// Block images per (b, h) unit that a chunked prefill reconstructs: the sink
// blocks holding tokens, then the tail's 32-token blocks.
static void prefill_blocks(const kvq_cache* c, int* nsb, int* nvb)
{
    const int n_sink = c->n < c->fmt.sink ? c->n : c->fmt.sink;
    const int tail = c->n > c->fmt.sink ? c->n - c->fmt.sink : 0;
    *nsb = (n_sink + 31) / 32;
    *nvb = *nsb + (tail + 31) / 32;
}

kvq_status kvq_prefill_workspace_bytes(const kvq_cache* c, size_t* bytes)
{
    if (!c || !bytes)
        return KVQ_ERR_ARG;
    int nsb, nvb;
    prefill_blocks(c, &nsb, &nvb);
    *bytes = (size_t)c->B * c->H * nvb * kvq::prefill_image_bytes(c->D);
    return KVQ_OK;
}

kvq_status kvq_prefill_attn(const kvq_cache* c, const void* Q, int C, int H_q, float sm_scale, void* O,
                            void* workspace, size_t ws_bytes, void* stream)
{
    if (!c || !Q || !O || !aligned16(Q) || !aligned16(O) || !isfinite(sm_scale))
        return KVQ_ERR_ARG;
    if (H_q < c->H || H_q % c->H != 0 || C < 1 || C > c->n)
        return KVQ_ERR_ARG;
    int nsb, nvb;
    prefill_blocks(c, &nsb, &nvb);
    if (!workspace || !aligned16(workspace) || ws_bytes < (size_t)nvb * kvq::prefill_image_bytes(c->D))
        return KVQ_ERR_WORKSPACE;
    const kvq_format& f = c->fmt;
    kvq::AttnParams p = {};
    p.nq = kvq::num_coded(f, c->n);
    p.kc = at<uint32_t>(c, 0);
    p.ks = at<float>(c, 1);
    p.kz = at<float>(c, 2);
    p.vc = at<uint32_t>(c, 3);
    p.vs = at<float>(c, 4);
    p.vz = at<float>(c, 5);
    p.kr = at<uint16_t>(c, 6);
    p.vr = at<uint16_t>(c, 7);
    p.kq = at<uint16_t>(c, 8);
    p.vq = at<uint16_t>(c, 9);
    p.q = (const uint16_t*)Q;
    p.out = (float*)O;
    p.B = c->B;
    p.H = c->H;
    p.H_q = H_q;
    p.G = H_q / c->H;
    p.T = c->T_alloc;
    // chunk positions are tail indices (token minus sink): the tail length
    // n - sink is negative when the cache ends inside the sink
    p.n = c->n - f.sink;
    p.C = C;
    p.ring = f.residual + f.flush;
    p.sink = f.sink;
    p.n_sink = c->n < f.sink ? c->n : f.sink;
    p.k_bits = f.k_bits;
    p.v_bits = f.v_bits;
    p.k_mode = f.k_mode;
    p.v_mode = f.v_mode;
    p.k_axis = f.k_axis;
    p.k_group = f.k_group;
    p.v_group = f.v_group;
    p.rotate = f.rotate;
    p.sm_log2 = sm_scale * 1.4426950408889634f;
    p.rot_c = rotation_constant(c->D);
    p.meta16 = f.meta_fp16;
    p.pf_ws = (uint8_t*)workspace;
    p.pf_nvb = nvb;
    p.pf_nsb = nsb;
    return kvq::launch_prefill(p, c->D, ws_bytes, (hipStream_t)stream) == hipSuccess ? KVQ_OK : KVQ_ERR_DEVICE;
}

}  // extern "C"
