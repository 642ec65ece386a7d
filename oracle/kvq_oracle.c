/*
 * kvq_oracle.c -- CPU oracle for the packed low-bit KV-cache decode path.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously correct
 * reference that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg load it.  It shares
 * no code, header, table or constant with the GPU library.
 *
 * Paper: "Quality Recovery for Quantized KV Caches via Low-Rank Attention
 * Adaptation" (Abdellatif).  What each entry point follows:
 *   orc_project       Sec. 3, Eq. (1)-(2) and Sec. 3.4 "Deployment overhead":
 *                     y_p = W_p h + (alpha/r) B_p (A_p h), in fp64.
 *   orc_merge_adapter Sec. 3.4 "Deployment overhead": the dense-base update
 *                     folded into the weights, W_p <- W_p + (alpha/r) B_p A_p.
 *   orc_quant_affine  Sec. 3.1 "Physical incremental cache", Eq. (3).
 *   orc_quant_sym     Sec. 3.1, the symmetric control (max-magnitude scale,
 *                     no offset); the exact formula is a reading (below).
 *   orc_quant_*16     the same with the metadata stored as fp16, as the
 *                     paper stores it (Sec. 3.1); rounding is a reading.
 *   orc_fwht_f32      Sec. 3.1, KVarN's fixed normalized Hadamard transform.
 *   orc_append        Sec. 3.1: new states are coded, packed and appended;
 *                     KIVI's fp16 residual window of recent tokens;
 *                     KVarN's fp16 sink tokens (the first S tokens).
 *   orc_dequant       Sec. 3.2: the reconstruction presented to attention.
 *   orc_decode_attn   Sec. 3.1-3.2: attention over that reconstruction, fp64.
 *   orc_prefill_attn  Sec. 3.1, chunked evaluation (128-token chunks): the
 *                     chunk's queries attend causally over the
 *                     reconstruction after the chunk has been appended.
 *
 * Arithmetic: the coding path (Eq. (3), the symmetric code, the Hadamard
 * butterflies) is IEEE binary32, one rounded operation at a time; the file
 * is compiled with -O2 -ffp-contract=off and no fast-math.  Projection,
 * reconstruction and attention accumulate in binary64.
 *
 * Threads: the loops over independent units -- (sequence, KV head) pairs
 * for append, reconstruction and attention, rows for the projection and
 * the merge -- are shared among OpenMP threads.  Each unit is still
 * computed by one thread in the serial order written below, so every
 * result is the same for any thread count (orc_set_threads).
 *
 * Storage image (the byte layout the GPU library must reproduce exactly):
 * sections Kc, Ks, Kz, Vc, Vs, Vz, Kr, Vr, Kq, Vq, each starting at a
 * multiple of 256 bytes.
 *
 * Sink tokens (a reading of KVarN's protected first tokens, Sec. 3.1): with
 * sink = S > 0 the first S tokens of a sequence are kept as fp16 rows
 * (rotated first when the format rotates) and never coded.  Tokens from S
 * on form the coded tail: tail token i is token S + i, and every rule below
 * (blocks, the residual window, the ring slot) applies to the tail indices
 * as it would to a cache without sinks.  Below, t is a tail index.
 *
 * T_alloc = max(T_max - S, 0) rounded up to a multiple of 32; NB =
 * T_alloc/32 blocks of 32 tokens per (b, h); u = b*H + h; token t is
 * position tau = t % 32 of block beta = t / 32.
 *
 * Codes are stored in pieces of eight codes, code j of a piece at bits
 * [bits*j, bits*j + bits) (a piece is a u64 for 8-bit codes, a u32 for
 * 4-bit codes, a u16 for 2-bit codes; piece i of a section starts at byte
 * i * bits).  The pieces of
 * a block are ordered for the consumer, a 64-lane MFMA layout: token tau has
 * row r = 4*(tau/8) + tau%4 in half e = (tau/4)%2 of its block.
 *   Kc  piece (t, P) = channels 8P..8P+7 of token t, P < D/8, at index
 *       (((u*NB + beta)*2 + e)*64 + r + 16*(P%4)) * (D/32) + P/4
 *   Vc  piece (o, d) = tokens 8o..8o+7 (octet o) of channel d, at index
 *       ((u*NB + o/4)*64 + d%16 + 16*(o%4)) * (D/16) + d/16
 *   Ks  per-token K scale of group g (channels g*kg ..), fp32 (fp16 when
 *       meta_fp16; element i at byte i*4 or i*2 of the section), at
 *       ((u*NB + beta)*(D/kg) + g)*32 + tau
 *       f32 per-channel K scale of (32-token group beta, channel d), at
 *       (u*NB + beta)*D + d
 *   Kz  like Ks, affine K only (zero bytes for symmetric K)
 *   Vs  per-token V scale of group g (fp32 or fp16 like Ks), at
 *       ((u*NB + beta)*(D/vg) + g)*32 + tau
 *   Vz  like Vs, affine V only
 *   Kr  f16 [B][H][R+F][D]             fp16 residual ring (F > 0 only)
 *   Vr  f16 [B][H][R+F][D]
 *   Kq  f16 [B][H][S][D]               fp16 sink tokens (S > 0 only)
 *   Vq  f16 [B][H][S][D]
 * The paper fixes the codes, their width and the metadata (Sec. 3.1), not
 * the order of the packed bytes; this order is the one the decode kernel
 * reads, so the packed cache is streamed without rearrangement.
 * orc_pack_word/orc_unpack_word pack a full 32-bit word (32/bits codes).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <omp.h>

enum {
    ORC_OK = 0,
    ORC_ERR_ARG = 1,
    ORC_ERR_FORMAT = 2,
    ORC_ERR_CAPACITY = 3,
    ORC_ERR_NONFINITE = 4,
    ORC_ERR_NOMEM = 5
};

typedef struct {
    int k_bits, v_bits;   /* 2 or 4 */
    int k_mode, v_mode;   /* 0 affine (Eq. (3)), 1 symmetric control */
    int k_axis, v_axis;   /* 0 groups along head_dim (per token), 1 groups of tokens (per channel, K only) */
    int k_group, v_group; /* group size: head_dim elements, or tokens for per-channel K */
    int residual, flush;  /* fp16 window: R newest tokens kept, flushed F at a time; 0,0 = none */
    int rotate;           /* 0, or head_dim: Hadamard rotation of K/V before coding */
    int meta_fp16;        /* 0: fp32 scales and offsets; 1: fp16 (the paper's storage) */
    int sink;             /* 0, or S (a multiple of 32): the first S tokens kept as fp16 */
} orc_format;

/* Threads used by the unit loops (n >= 1), and the current setting. */
void orc_set_threads(int n)
{
    if (n >= 1)
        omp_set_num_threads(n);
}

int orc_get_threads(void)
{
    return omp_get_max_threads();
}

/* ------------------------------------------------------------------ */
/* Scalar number formats                                               */
/* ------------------------------------------------------------------ */

static float bf16_to_f32(uint16_t h)
{
    uint32_t x = (uint32_t)h << 16;
    float f;
    memcpy(&f, &x, 4);
    return f;
}

/* Round a finite non-negative value to the grid {r * 2^q : r integer} with
 * ties to even r.  Dividing by a power of two is exact in binary64. */
static double round_to_grid(double a, int q)
{
    return rint(ldexp(a, -q));
}

/* binary32 -> binary16, round to nearest, ties to even.  binary16 has an
 * 11-bit significand, exponents -14..15 and subnormal spacing 2^-24; a
 * value that rounds to 2^16 or more overflows to infinity. */
uint16_t orc_f32_to_f16(float f)
{
    uint16_t sign = signbit(f) ? 0x8000 : 0;
    double a = fabs((double)f);
    if (isnan(f))
        return sign | 0x7e00;
    if (isinf(f))
        return sign | 0x7c00;
    int ex;
    frexp(a, &ex);                 /* 2^(ex-1) <= a < 2^ex */
    int e = ex - 1;
    if (a == 0.0 || e < -14) {     /* subnormal range: spacing 2^-24 */
        double r = round_to_grid(a, -24);
        return sign | (uint16_t)r; /* r == 1024 encodes 2^-14 exactly */
    }
    if (e > 15)
        return sign | 0x7c00;
    double r = round_to_grid(a, e - 10); /* r in [1024, 2048] */
    if (r * ldexp(1.0, e - 10) >= 65536.0)
        return sign | 0x7c00;
    return sign | (uint16_t)(((e + 15) << 10) + ((int)r - 1024));
}

float orc_f16_to_f32(uint16_t h)
{
    int ex = (h >> 10) & 31, m = h & 1023;
    double v;
    if (ex == 0)
        v = ldexp((double)m, -24);
    else if (ex == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + m), ex - 25);
    return (float)((h & 0x8000) ? -v : v);
}

/* binary64 -> bfloat16, round to nearest, ties to even (8-bit significand,
 * binary32 exponent range, subnormal spacing 2^-133). */
uint16_t orc_f64_to_bf16(double y)
{
    uint16_t sign = signbit(y) ? 0x8000 : 0;
    double a = fabs(y);
    if (isnan(y))
        return sign | 0x7fc0;
    if (isinf(y))
        return sign | 0x7f80;
    int ex;
    frexp(a, &ex);
    int e = ex - 1;
    if (a == 0.0 || e < -126) {
        double r = round_to_grid(a, -133);
        return sign | (uint16_t)r;
    }
    if (e > 127)
        return sign | 0x7f80;
    double r = round_to_grid(a, e - 7); /* r in [128, 256] */
    if (r * ldexp(1.0, e - 7) >= ldexp(1.0, 128))
        return sign | 0x7f80;
    return sign | (uint16_t)(((e + 127) << 7) + ((int)r - 128));
}

/* ------------------------------------------------------------------ */
/* Grouped codes (Sec. 3.1)                                             */
/* ------------------------------------------------------------------ */

/* Eq. (3), one group of g values:
 *   s = max((max x - min x) / (2^b - 1), 1e-8)
 *   c = clip(round((x - min x) / s), 0, 2^b - 1)
 * round() is half-to-even (the paper leaves the tie rule unstated).  The
 * offset stored beside the scale is min x itself (a float, not an integer
 * zero point); a signed zero is stored as +0.0 so the metadata does not
 * depend on which of two equal zeros a reduction meets first. */
void orc_quant_affine(const float* x, int g, int bits, uint8_t* codes, float* s_out, float* z_out)
{
    float mn = x[0], mx = x[0];
    for (int i = 1; i < g; ++i) {
        if (x[i] < mn)
            mn = x[i];
        if (x[i] > mx)
            mx = x[i];
    }
    const float top = (float)((1 << bits) - 1);
    float range = mx - mn;
    float s = range / top;
    if (!(s >= 1e-8f))
        s = 1e-8f;
    for (int i = 0; i < g; ++i) {
        float d = x[i] - mn;
        float c = rintf(d / s);
        if (c < 0.0f)
            c = 0.0f;
        if (c > top)
            c = top;
        codes[i] = (uint8_t)c;
    }
    *s_out = s;
    *z_out = mn + 0.0f;
}

/* Symmetric control (Sec. 3.1: maximum-magnitude scale, no offset).
 * Reading: qmax = 2^(b-1) - 1, s = max(max|x| / qmax, 1e-8),
 * q = clip(round(x / s), -qmax, qmax) with half-to-even rounding, and the
 * unsigned code stored is u = q + 2^(b-1) (so u is in [1, 2^b - 1]).
 * Reconstruction is (u - 2^(b-1)) * s. */
void orc_quant_sym(const float* x, int g, int bits, uint8_t* codes, float* s_out)
{
    float ma = 0.0f;
    for (int i = 0; i < g; ++i) {
        float a = fabsf(x[i]);
        if (a > ma)
            ma = a;
    }
    const float qmax = (float)((1 << (bits - 1)) - 1);
    float s = ma / qmax;
    if (!(s >= 1e-8f))
        s = 1e-8f;
    for (int i = 0; i < g; ++i) {
        float q = rintf(x[i] / s);
        if (q < -qmax)
            q = -qmax;
        if (q > qmax)
            q = qmax;
        codes[i] = (uint8_t)(int)(q + (float)(1 << (bits - 1)));
    }
    *s_out = s;
}

/* fp16 metadata (Sec. 3.1 keeps each group's scale and offset in fp16).
 * Reading: the scale and offset are computed in fp32 exactly as above, then
 * rounded to fp16 (nearest, ties to even), the scale first clamped to
 * [2^-24, 65504] (the 1e-8 floor lies below fp16's smallest subnormal) and
 * the offset to [-65504, 65504]; the codes are then computed from the
 * rounded values, so they are the best codes for the metadata actually
 * stored.  s16 / z16 receive the fp16 bit patterns. */
static float to_f16_value(float v, float lo, float hi)
{
    if (v < lo)
        v = lo;
    if (v > hi)
        v = hi;
    return orc_f16_to_f32(orc_f32_to_f16(v));
}

void orc_quant_affine16(const float* x, int g, int bits, uint8_t* codes, uint16_t* s16, uint16_t* z16)
{
    float s, z;
    orc_quant_affine(x, g, bits, codes, &s, &z);
    s = to_f16_value(s, 0x1p-24f, 65504.0f);
    z = to_f16_value(z, -65504.0f, 65504.0f) + 0.0f;
    const float top = (float)((1 << bits) - 1);
    for (int i = 0; i < g; ++i) {
        float c = rintf((x[i] - z) / s);
        if (c < 0.0f)
            c = 0.0f;
        if (c > top)
            c = top;
        codes[i] = (uint8_t)c;
    }
    *s16 = orc_f32_to_f16(s);
    *z16 = orc_f32_to_f16(z);
}

void orc_quant_sym16(const float* x, int g, int bits, uint8_t* codes, uint16_t* s16)
{
    float s;
    orc_quant_sym(x, g, bits, codes, &s);
    s = to_f16_value(s, 0x1p-24f, 65504.0f);
    const float qmax = (float)((1 << (bits - 1)) - 1);
    for (int i = 0; i < g; ++i) {
        float q = rintf(x[i] / s);
        if (q < -qmax)
            q = -qmax;
        if (q > qmax)
            q = qmax;
        codes[i] = (uint8_t)(int)(q + (float)(1 << (bits - 1)));
    }
    *s16 = orc_f32_to_f16(s);
}

/* Packing: the run c[0..32/b) goes into one little-endian 32-bit word,
 * element j at bits [b*j, b*j + b). */
uint32_t orc_pack_word(const uint8_t* codes, int bits)
{
    uint32_t w = 0;
    for (int j = 0; j < 32 / bits; ++j)
        w |= (uint32_t)codes[j] << (bits * j);
    return w;
}

void orc_unpack_word(uint32_t w, int bits, uint8_t* codes)
{
    for (int j = 0; j < 32 / bits; ++j)
        codes[j] = (uint8_t)((w >> (bits * j)) & ((1u << bits) - 1));
}

/* ------------------------------------------------------------------ */
/* Hadamard rotation (Sec. 3.1, KVarN format)                          */
/* ------------------------------------------------------------------ */

/* Fixed normalized Walsh-Hadamard transform of n (a power of two) values,
 * in binary32: radix-2 butterflies with half-width h = 1, 2, 4, ..., n/2,
 * each pair (x_j, x_{j+h}) -> (x_j + x_{j+h}, x_j - x_{j+h}) for j in the
 * lower half of each block of 2h, then one multiply by the binary32 value
 * nearest n^(-1/2).  The result is (1/sqrt(n)) H_n x with H_n the Sylvester
 * matrix; the stage order fixes the rounding so coded values are exact. */
void orc_fwht_f32(float* x, int n)
{
    for (int h = 1; h < n; h *= 2) {
        for (int blk = 0; blk < n; blk += 2 * h) {
            for (int j = blk; j < blk + h; ++j) {
                float a = x[j], b = x[j + h];
                x[j] = a + b;
                x[j + h] = a - b;
            }
        }
    }
    const float c = (float)(1.0 / sqrt((double)n));
    for (int j = 0; j < n; ++j)
        x[j] = x[j] * c;
}

/* Sylvester Hadamard entry: H[i][j] = (-1)^popcount(i & j). */
static double hadamard_entry(int i, int j)
{
    unsigned v = (unsigned)(i & j);
    int parity = 0;
    while (v) {
        parity ^= (int)(v & 1u);
        v >>= 1;
    }
    return parity ? -1.0 : 1.0;
}

/* y = (1/sqrt(n)) H_n x in binary64, from the matrix definition. */
static void rotate_f64(const double* x, double* y, int n)
{
    const double c = 1.0 / sqrt((double)n);
    for (int i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int j = 0; j < n; ++j)
            acc += hadamard_entry(i, j) * x[j];
        y[i] = c * acc;
    }
}

/* ------------------------------------------------------------------ */
/* Cache format and storage image                                       */
/* ------------------------------------------------------------------ */

static int is_pow2_in(int v, int lo, int hi)
{
    return v >= lo && v <= hi && (v & (v - 1)) == 0;
}

int orc_check_format(const orc_format* f, int D)
{
    if (!f)
        return ORC_ERR_ARG;
    if (D != 64 && D != 128 && D != 256)
        return ORC_ERR_FORMAT;
    if ((f->k_bits != 2 && f->k_bits != 4 && f->k_bits != 8) || (f->v_bits != 2 && f->v_bits != 4 && f->v_bits != 8))
        return ORC_ERR_FORMAT;
    if ((f->k_mode != 0 && f->k_mode != 1) || (f->v_mode != 0 && f->v_mode != 1))
        return ORC_ERR_FORMAT;
    if ((f->k_axis != 0 && f->k_axis != 1) || f->v_axis != 0)
        return ORC_ERR_FORMAT;
    if (f->residual < 0 || f->flush < 0 || (f->flush == 0 && f->residual != 0))
        return ORC_ERR_FORMAT;
    if (f->flush % 32 != 0)
        return ORC_ERR_FORMAT;
    if (f->rotate != 0 && f->rotate != D)
        return ORC_ERR_FORMAT;
    if (f->k_axis == 0) {
        if (!is_pow2_in(f->k_group, 32, D))
            return ORC_ERR_FORMAT;
    } else {
        if (f->k_group != 32 || f->flush == 0)
            return ORC_ERR_FORMAT;
    }
    if (!is_pow2_in(f->v_group, 32, D))
        return ORC_ERR_FORMAT;
    if (f->meta_fp16 != 0 && f->meta_fp16 != 1)
        return ORC_ERR_FORMAT;
    if (f->sink < 0 || f->sink % 32 != 0)
        return ORC_ERR_FORMAT;
    return ORC_OK;
}

static size_t round_up(size_t v, size_t a)
{
    return (v + a - 1) / a * a;
}

/* Tail slots allocated per (b, h): T_max - S rounded up to 32. */
static size_t tail_alloc(const orc_format* f, int T_max)
{
    return T_max > f->sink ? round_up((size_t)(T_max - f->sink), 32) : 0;
}

/* Byte offsets and lengths of the ten sections; see the file header. */
int orc_layout(const orc_format* f, int B, int H, int D, int T_max, size_t off[10], size_t len[10], size_t* total)
{
    int st = orc_check_format(f, D);
    if (st)
        return st;
    if (B < 1 || H < 1 || T_max < 1)
        return ORC_ERR_ARG;
    size_t bh = (size_t)B * H;
    size_t T = tail_alloc(f, T_max);
    size_t ring = (size_t)(f->residual + f->flush);
    len[0] = bh * T * (size_t)(D * f->k_bits / 32) * 4;
    const size_t msz = f->meta_fp16 ? 2 : 4; /* bytes per scale or offset */
    if (f->k_axis == 0)
        len[1] = bh * T * (size_t)(D / f->k_group) * msz;
    else
        len[1] = bh * (T / 32) * (size_t)D * msz;
    len[2] = f->k_mode == 0 ? len[1] : 0;
    len[3] = bh * (T * f->v_bits / 32) * (size_t)D * 4;
    len[4] = bh * T * (size_t)(D / f->v_group) * msz;
    len[5] = f->v_mode == 0 ? len[4] : 0;
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
    return ORC_OK;
}

/* Tokens held as codes when n tokens are cached, counted over the tail of
 * m = max(0, n - S) tokens after the sink: all m without a residual window,
 * else floor(max(0, m - R) / F) * F (the newest R..R+F-1 stay fp16). */
int orc_num_coded(const orc_format* f, int n)
{
    n = n > f->sink ? n - f->sink : 0;
    if (f->flush == 0)
        return n;
    int over = n - f->residual;
    if (over <= 0)
        return 0;
    return over / f->flush * f->flush;
}

typedef struct {
    const orc_format* f;
    int B, H, D, T;     /* T = T_alloc */
    uint8_t* img;
    size_t off[10];
} image_view;

static int view_init(image_view* v, const orc_format* f, int B, int H, int D, int T_max, const uint8_t* img)
{
    size_t len[10], total;
    int st = orc_layout(f, B, H, D, T_max, v->off, len, &total);
    if (st)
        return st;
    v->f = f;
    v->B = B;
    v->H = H;
    v->D = D;
    v->T = (int)tail_alloc(f, T_max);
    v->img = (uint8_t*)img;
    return ORC_OK;
}

static size_t unit_block(const image_view* v, int b, int h, int t)
{
    return ((size_t)b * v->H + h) * (size_t)(v->T / 32) + (size_t)(t / 32);
}

/* Score-row of position tau in its half block, and the half. */
static int row_of(int tau) { return 4 * (tau / 8) + tau % 4; }
static int half_of(int tau) { return (tau / 4) % 2; }

/* Byte address of K piece P (channels 8P..8P+7) of token t. */
static uint8_t* kc_piece(const image_view* v, int b, int h, int t, int P)
{
    int tau = t % 32;
    size_t lane = (size_t)row_of(tau) + 16 * (size_t)(P % 4);
    size_t i = ((unit_block(v, b, h, t) * 2 + (size_t)half_of(tau)) * 64 + lane) * (size_t)(v->D / 32) + (size_t)(P / 4);
    return v->img + v->off[0] + i * (size_t)v->f->k_bits;
}

/* Byte address of V piece (octet t / 8, channel d). */
static uint8_t* vc_piece(const image_view* v, int b, int h, int t, int d)
{
    int o = (t % 32) / 8;
    size_t lane = (size_t)(d % 16) + 16 * (size_t)o;
    size_t i = (unit_block(v, b, h, t) * 64 + lane) * (size_t)(v->D / 16) + (size_t)(d / 16);
    return v->img + v->off[3] + i * (size_t)v->f->v_bits;
}

/* A piece holds eight codes of `bits` bits: 64 bits for 8-bit codes, 32 for
 * 4-bit, 16 for 2-bit (little-endian, code j at bits [bits*j, +bits)). */
static uint64_t piece_get(const uint8_t* p, int bits)
{
    uint64_t w = 0;
    memcpy(&w, p, (size_t)bits);
    return w;
}

static void piece_put(uint8_t* p, int bits, uint64_t val)
{
    memcpy(p, &val, (size_t)bits);
}

static uint64_t pack8(const uint8_t* codes, int bits)
{
    uint64_t w = 0;
    for (int j = 0; j < 8; ++j)
        w |= (uint64_t)codes[j] << (bits * j);
    return w;
}

/* Index of K metadata for (b, h, token t, head_dim element d). */
static size_t kmeta_index(const image_view* v, int b, int h, int t, int d)
{
    if (v->f->k_axis == 0) {
        size_t gpt = (size_t)(v->D / v->f->k_group);
        return (unit_block(v, b, h, t) * gpt + (size_t)(d / v->f->k_group)) * 32 + (size_t)(t % 32);
    }
    return unit_block(v, b, h, t) * v->D + d;
}

static size_t vmeta_index(const image_view* v, int b, int h, int t, int d)
{
    size_t gpt = (size_t)(v->D / v->f->v_group);
    return (unit_block(v, b, h, t) * gpt + (size_t)(d / v->f->v_group)) * 32 + (size_t)(t % 32);
}

static uint16_t* ring_entry(const image_view* v, int which, int b, int h, int t)
{
    int R = v->f->residual + v->f->flush;
    size_t i = (((size_t)b * v->H + h) * R + (size_t)(t % R)) * v->D;
    return (uint16_t*)(v->img + v->off[which ? 7 : 6]) + i;
}

/* fp16 row of sink token t (t < S). */
static uint16_t* sink_entry(const image_view* v, int which, int b, int h, int t)
{
    size_t i = (((size_t)b * v->H + h) * (size_t)v->f->sink + (size_t)t) * v->D;
    return (uint16_t*)(v->img + v->off[which ? 9 : 8]) + i;
}

/* Scale or offset i of a metadata section (1, 2, 4, 5), fp32 or fp16. */
static float meta_get(const image_view* v, int section, size_t i)
{
    if (v->f->meta_fp16) {
        uint16_t h;
        memcpy(&h, v->img + v->off[section] + 2 * i, 2);
        return orc_f16_to_f32(h);
    }
    float x;
    memcpy(&x, v->img + v->off[section] + 4 * i, 4);
    return x;
}

/* Store a value that the section's precision represents exactly. */
static void meta_put(const image_view* v, int section, size_t i, float x)
{
    if (v->f->meta_fp16) {
        uint16_t h = orc_f32_to_f16(x);
        memcpy(v->img + v->off[section] + 2 * i, &h, 2);
    } else {
        memcpy(v->img + v->off[section] + 4 * i, &x, 4);
    }
}

/* ------------------------------------------------------------------ */
/* Append (Sec. 3.1: new states are packed and appended)                */
/* ------------------------------------------------------------------ */

/* The D values of tail token t, (b, h), for K (which = 0) or V (which = 1),
 * as the coder sees them: the bf16 input (rotated in binary32 when the
 * format rotates); with a residual window, rounded to fp16, or read back
 * from the fp16 ring for tokens appended by an earlier call.  n0 is the tail
 * index of the call's first input token (negative when the call starts in
 * the sink). */
static void token_values(const image_view* v, int which, const uint16_t* X, int n0, int n_new, int b, int h, int t,
                         float* out)
{
    const orc_format* f = v->f;
    int D = v->D;
    if (t >= n0) {
        const uint16_t* src = X + (((size_t)b * n_new + (t - n0)) * v->H + h) * D;
        for (int d = 0; d < D; ++d)
            out[d] = bf16_to_f32(src[d]);
        if (f->rotate)
            orc_fwht_f32(out, D);
        if (f->flush)
            for (int d = 0; d < D; ++d)
                out[d] = orc_f16_to_f32(orc_f32_to_f16(out[d]));
    } else {
        const uint16_t* r = ring_entry(v, which, b, h, t);
        for (int d = 0; d < D; ++d)
            out[d] = orc_f16_to_f32(r[d]);
    }
}

static void code_group(int mode, int bits, int meta16, const float* x, int g, uint8_t* codes, float* s, float* z)
{
    if (meta16) {
        uint16_t s16, z16 = 0;
        if (mode == 0)
            orc_quant_affine16(x, g, bits, codes, &s16, &z16);
        else
            orc_quant_sym16(x, g, bits, codes, &s16);
        *s = orc_f16_to_f32(s16);
        *z = orc_f16_to_f32(z16);
        return;
    }
    if (mode == 0) {
        orc_quant_affine(x, g, bits, codes, s, z);
    } else {
        orc_quant_sym(x, g, bits, codes, s);
        *z = 0.0f;
    }
}

/* Append n_new tokens.  K and V are bf16 [B][n_new][H][D].  On success the
 * image holds, for every token t below the new length n, the codes and
 * metadata of t (tokens below the coded count) and the fp16 ring holds the
 * newest R + F tokens.  The result depends only on the tokens appended so
 * far, not on how they were split into calls.  Errors change nothing. */
int orc_append(const orc_format* f, int B, int H, int D, int T_max, uint8_t* image, int* n_io, const uint16_t* K,
               const uint16_t* V, int n_new)
{
    image_view v;
    int st = view_init(&v, f, B, H, D, T_max, image);
    if (st)
        return st;
    if (!n_io || n_new < 0 || (n_new > 0 && (!K || !V)))
        return ORC_ERR_ARG;
    int n0 = *n_io, n1 = n0 + n_new;
    if (n0 < 0 || n1 > T_max)
        return ORC_ERR_CAPACITY;
    size_t count = (size_t)B * n_new * H * D;
    for (size_t i = 0; i < count; ++i)
        if (!isfinite(bf16_to_f32(K[i])) || !isfinite(bf16_to_f32(V[i])))
            return ORC_ERR_NONFINITE;

    /* sink tokens [n0, min(S, n1)); tail indices [n0t, n1t) for the rest */
    const int S = f->sink, n0t = n0 - S, n1t = n1 - S;
    const int q0 = orc_num_coded(f, n0), q1 = orc_num_coded(f, n1);
    const int kb = f->k_bits, vb = f->v_bits;
    const int m16 = f->meta_fp16;
    int nomem = 0;

    /* (b, h) units are independent: each writes only its own pieces,
     * metadata and rows. */
#pragma omp parallel reduction(| : nomem)
    {
    float* x = (float*)malloc(sizeof(float) * (size_t)D * 32);
    uint8_t* codes = (uint8_t*)malloc((size_t)D * 32);
    if (!x || !codes)
        nomem = 1;
#pragma omp for schedule(dynamic, 1)
    for (int u = 0; u < B * H; ++u) {
        if (!x || !codes)
            continue;
        const int b = u / H, h = u % H;
        {
            /* K, groups along head_dim: each coded token on its own. */
            if (f->k_axis == 0) {
                for (int t = q0; t < q1; ++t) {
                    token_values(&v, 0, K, n0t, n_new, b, h, t, x);
                    for (int d0 = 0; d0 < D; d0 += f->k_group) {
                        float s, z;
                        code_group(f->k_mode, kb, m16, x + d0, f->k_group, codes + d0, &s, &z);
                        size_t mi = kmeta_index(&v, b, h, t, d0);
                        meta_put(&v, 1, mi, s);
                        if (f->k_mode == 0)
                            meta_put(&v, 2, mi, z);
                    }
                    for (int P = 0; P < D / 8; ++P)
                        piece_put(kc_piece(&v, b, h, t, P), kb, pack8(codes + 8 * P, kb));
                }
            } else {
                /* K, groups of 32 tokens per channel (KIVI keys). */
                for (int t0 = q0; t0 < q1; t0 += 32) {
                    for (int i = 0; i < 32; ++i)
                        token_values(&v, 0, K, n0t, n_new, b, h, t0 + i, x + (size_t)i * D);
                    float col[32];
                    uint8_t cc[32];
                    for (int d = 0; d < D; ++d) {
                        float s, z;
                        for (int i = 0; i < 32; ++i)
                            col[i] = x[(size_t)i * D + d];
                        code_group(f->k_mode, kb, m16, col, 32, cc, &s, &z);
                        size_t mi = kmeta_index(&v, b, h, t0, d);
                        meta_put(&v, 1, mi, s);
                        if (f->k_mode == 0)
                            meta_put(&v, 2, mi, z);
                        for (int i = 0; i < 32; ++i)
                            codes[(size_t)i * D + d] = cc[i];
                    }
                    for (int i = 0; i < 32; ++i)
                        for (int P = 0; P < D / 8; ++P)
                            piece_put(kc_piece(&v, b, h, t0 + i, P), kb, pack8(codes + (size_t)i * D + 8 * P, kb));
                }
            }
            /* V, groups along head_dim; codes packed along tokens.  Writing
             * token t keeps the bits of earlier tokens in its piece and
             * clears those of t and later tokens before inserting t's code. */
            for (int t = q0; t < q1; ++t) {
                token_values(&v, 1, V, n0t, n_new, b, h, t, x);
                for (int d0 = 0; d0 < D; d0 += f->v_group) {
                    float s, z;
                    code_group(f->v_mode, vb, m16, x + d0, f->v_group, codes + d0, &s, &z);
                    size_t mi = vmeta_index(&v, b, h, t, d0);
                    meta_put(&v, 4, mi, s);
                    if (f->v_mode == 0)
                        meta_put(&v, 5, mi, z);
                }
                int j = t % 8;
                uint64_t keep = j == 0 ? 0u : ((1ull << (vb * j)) - 1u);
                for (int d = 0; d < D; ++d) {
                    uint8_t* pc = vc_piece(&v, b, h, t, d);
                    piece_put(pc, vb, (piece_get(pc, vb) & keep) | ((uint64_t)codes[d] << (vb * j)));
                }
            }
            /* sink tokens: the fp16 of the (rotated) input, row t */
            for (int which = 0; which < 2; ++which) {
                for (int t = n0; t < n1 && t < S; ++t) {
                    const uint16_t* src = (which ? V : K) + (((size_t)b * n_new + (t - n0)) * H + h) * D;
                    for (int d = 0; d < D; ++d)
                        x[d] = bf16_to_f32(src[d]);
                    if (f->rotate)
                        orc_fwht_f32(x, D);
                    uint16_t* r = sink_entry(&v, which, b, h, t);
                    for (int d = 0; d < D; ++d)
                        r[d] = orc_f32_to_f16(x[d]);
                }
            }
            /* fp16 residual ring: slot t mod (R + F) holds the newest token
             * with that residue (written after the coder has read it). */
            if (f->flush) {
                int ring = f->residual + f->flush;
                int t_lo = n0t > 0 ? n0t : 0;
                if (n1t - ring > t_lo)
                    t_lo = n1t - ring;
                for (int which = 0; which < 2; ++which) {
                    for (int t = t_lo; t < n1t; ++t) {
                        token_values(&v, which, which ? V : K, n0t, n_new, b, h, t, x);
                        uint16_t* r = ring_entry(&v, which, b, h, t);
                        for (int d = 0; d < D; ++d)
                            r[d] = orc_f32_to_f16(x[d]);
                    }
                }
            }
        }
    }
    free(x);
    free(codes);
    }
    if (nomem)
        return ORC_ERR_NOMEM;
    *n_io = n1;
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Reconstruction and attention (Sec. 3.1-3.2)                          */
/* ------------------------------------------------------------------ */

static double dequant_code(int mode, int bits, uint32_t c, float s, float z)
{
    if (mode == 0)
        return (double)c * (double)s + (double)z;
    return ((double)c - (double)(1 << (bits - 1))) * (double)s;
}

/* Reconstruction of tokens [0, n) of (b, h) into khat, vhat [n][D] (fp64):
 * sink tokens from their fp16 rows; tail token i = t - S from codes and
 * metadata while i is below the coded count, else from the fp16 ring.
 * Values stay in the rotated basis when the format rotates. */
static void reconstruct_bh(const image_view* v, int b, int h, int n, double* khat, double* vhat)
{
    const orc_format* f = v->f;
    int D = v->D, nq = orc_num_coded(f, n), S = f->sink;
    const int kb = f->k_bits, vb = f->v_bits;
    for (int t = 0; t < n; ++t) {
        const int i = t - S; /* tail index */
        for (int d = 0; d < D; ++d) {
            double kv, vv;
            if (t < S) {
                kv = orc_f16_to_f32(sink_entry(v, 0, b, h, t)[d]);
                vv = orc_f16_to_f32(sink_entry(v, 1, b, h, t)[d]);
            } else if (i < nq) {
                uint64_t kw = piece_get(kc_piece(v, b, h, i, d / 8), kb);
                uint32_t kc = (uint32_t)(kw >> (kb * (d % 8))) & ((1u << kb) - 1u);
                size_t km = kmeta_index(v, b, h, i, d);
                kv = dequant_code(f->k_mode, kb, kc, meta_get(v, 1, km), f->k_mode == 0 ? meta_get(v, 2, km) : 0.0f);
                uint64_t vw = piece_get(vc_piece(v, b, h, i, d), vb);
                uint32_t vc = (uint32_t)(vw >> (vb * (i % 8))) & ((1u << vb) - 1u);
                size_t vm = vmeta_index(v, b, h, i, d);
                vv = dequant_code(f->v_mode, vb, vc, meta_get(v, 4, vm), f->v_mode == 0 ? meta_get(v, 5, vm) : 0.0f);
            } else {
                kv = orc_f16_to_f32(ring_entry(v, 0, b, h, i)[d]);
                vv = orc_f16_to_f32(ring_entry(v, 1, b, h, i)[d]);
            }
            khat[(size_t)t * D + d] = kv;
            vhat[(size_t)t * D + d] = vv;
        }
    }
}

/* Reconstructed cache, Khat and Vhat [B][H][n][D] fp64. */
int orc_dequant(const orc_format* f, int B, int H, int D, int T_max, const uint8_t* image, int n, double* Khat,
                double* Vhat)
{
    image_view v;
    int st = view_init(&v, f, B, H, D, T_max, image);
    if (st)
        return st;
    if (n < 0 || n > T_max)
        return ORC_ERR_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < B * H; ++u) {
        size_t o = (size_t)u * (size_t)n * D;
        reconstruct_bh(&v, u / H, u % H, n, Khat + o, Vhat + o);
    }
    return ORC_OK;
}

/* Decode attention for one new query per sequence.  Q is bf16 [B][H_q][D],
 * O is fp64 [B][H_q][D].  Query head hq reads KV head hq / (H_q / H)
 * (contiguous grouped-query mapping, a reading).  For each head:
 *   l_t = sm * (q . khat_t),  p = softmax(l) (max-subtracted),
 *   o = sum_t p_t vhat_t.
 * With a rotating format, q is rotated first and o is rotated back (the
 * normalized Sylvester transform is its own inverse). */
int orc_decode_attn(const orc_format* f, int B, int H, int D, int T_max, const uint8_t* image, int n,
                    const uint16_t* Q, int H_q, double sm, double* O)
{
    image_view v;
    int st = view_init(&v, f, B, H, D, T_max, image);
    if (st)
        return st;
    if (n < 1 || n > T_max || H_q < H || H_q % H != 0 || !Q || !O)
        return ORC_ERR_ARG;
    const int G = H_q / H;
    int nomem = 0;
    /* (b, KV head) units are independent; each thread has its own buffers. */
#pragma omp parallel reduction(| : nomem)
    {
    double* khat = (double*)malloc(sizeof(double) * (size_t)n * D);
    double* vhat = (double*)malloc(sizeof(double) * (size_t)n * D);
    double* logit = (double*)malloc(sizeof(double) * (size_t)n);
    double* q = (double*)malloc(sizeof(double) * (size_t)D * 2);
    const int ok = khat && vhat && logit && q;
    if (!ok)
        nomem = 1;
    double* o = ok ? q + D : NULL;
#pragma omp for schedule(dynamic, 1)
    for (int u = 0; u < B * H; ++u) {
        if (!ok)
            continue;
        const int b = u / H, h = u % H;
        {
            reconstruct_bh(&v, b, h, n, khat, vhat);
            for (int hq = h * G; hq < (h + 1) * G; ++hq) {
                const uint16_t* qs = Q + ((size_t)b * H_q + hq) * D;
                for (int d = 0; d < D; ++d)
                    o[d] = bf16_to_f32(qs[d]);
                if (f->rotate)
                    rotate_f64(o, q, D);
                else
                    memcpy(q, o, sizeof(double) * (size_t)D);
                double mx = -INFINITY;
                for (int t = 0; t < n; ++t) {
                    double acc = 0.0;
                    for (int d = 0; d < D; ++d)
                        acc += q[d] * khat[(size_t)t * D + d];
                    logit[t] = sm * acc;
                    if (logit[t] > mx)
                        mx = logit[t];
                }
                double z = 0.0;
                for (int t = 0; t < n; ++t) {
                    logit[t] = exp(logit[t] - mx);
                    z += logit[t];
                }
                for (int d = 0; d < D; ++d)
                    o[d] = 0.0;
                for (int t = 0; t < n; ++t) {
                    double p = logit[t] / z;
                    for (int d = 0; d < D; ++d)
                        o[d] += p * vhat[(size_t)t * D + d];
                }
                double* dst = O + ((size_t)b * H_q + hq) * D;
                if (f->rotate)
                    rotate_f64(o, dst, D);
                else
                    memcpy(dst, o, sizeof(double) * (size_t)D);
            }
        }
    }
    free(khat);
    free(vhat);
    free(logit);
    free(q);
    }
    return nomem ? ORC_ERR_NOMEM : ORC_OK;
}

/* Chunked prefill attention (Sec. 3.1: evaluation runs chunk by chunk; the
 * chunk's states are coded and appended, then the reconstruction feeds
 * attention).  The cache holds n tokens, the last C of which are the
 * chunk; Q is bf16 [B][C][H_q][D] for positions n - C .. n - 1 and O is fp64
 * [B][C][H_q][D].  Query i of the chunk (position n - C + i) attends to the
 * reconstructed tokens 0 .. n - C + i (causal), otherwise exactly as
 * orc_decode_attn: max-subtracted softmax of sm * (q . khat_t), q rotated
 * first and o rotated back when the format rotates.  C = 1 is the decode
 * attention of the newest token. */
int orc_prefill_attn(const orc_format* f, int B, int H, int D, int T_max, const uint8_t* image, int n, int C,
                     const uint16_t* Q, int H_q, double sm, double* O)
{
    image_view v;
    int st = view_init(&v, f, B, H, D, T_max, image);
    if (st)
        return st;
    if (n < 1 || n > T_max || C < 1 || C > n || H_q < H || H_q % H != 0 || !Q || !O)
        return ORC_ERR_ARG;
    const int G = H_q / H;
    int nomem = 0;
    /* (b, KV head) units are independent; each thread has its own buffers. */
#pragma omp parallel reduction(| : nomem)
    {
    double* khat = (double*)malloc(sizeof(double) * (size_t)n * D);
    double* vhat = (double*)malloc(sizeof(double) * (size_t)n * D);
    double* logit = (double*)malloc(sizeof(double) * (size_t)n);
    double* q = (double*)malloc(sizeof(double) * (size_t)D * 2);
    const int ok = khat && vhat && logit && q;
    if (!ok)
        nomem = 1;
    double* o = ok ? q + D : NULL;
#pragma omp for schedule(dynamic, 1)
    for (int u = 0; u < B * H; ++u) {
        if (!ok)
            continue;
        const int b = u / H, h = u % H;
        {
            reconstruct_bh(&v, b, h, n, khat, vhat);
            for (int i = 0; i < C; ++i) {
                const int last = n - C + i;  /* newest token this query sees */
                for (int hq = h * G; hq < (h + 1) * G; ++hq) {
                    const uint16_t* qs = Q + (((size_t)b * C + i) * H_q + hq) * D;
                    for (int d = 0; d < D; ++d)
                        o[d] = bf16_to_f32(qs[d]);
                    if (f->rotate)
                        rotate_f64(o, q, D);
                    else
                        memcpy(q, o, sizeof(double) * (size_t)D);
                    double mx = -INFINITY;
                    for (int t = 0; t <= last; ++t) {
                        double acc = 0.0;
                        for (int d = 0; d < D; ++d)
                            acc += q[d] * khat[(size_t)t * D + d];
                        logit[t] = sm * acc;
                        if (logit[t] > mx)
                            mx = logit[t];
                    }
                    double z = 0.0;
                    for (int t = 0; t <= last; ++t) {
                        logit[t] = exp(logit[t] - mx);
                        z += logit[t];
                    }
                    for (int d = 0; d < D; ++d)
                        o[d] = 0.0;
                    for (int t = 0; t <= last; ++t) {
                        double p = logit[t] / z;
                        for (int d = 0; d < D; ++d)
                            o[d] += p * vhat[(size_t)t * D + d];
                    }
                    double* dst = O + (((size_t)b * C + i) * H_q + hq) * D;
                    if (f->rotate)
                        rotate_f64(o, dst, D);
                    else
                        memcpy(dst, o, sizeof(double) * (size_t)D);
                }
            }
        }
    }
    free(khat);
    free(vhat);
    free(logit);
    free(q);
    }
    return nomem ? ORC_ERR_NOMEM : ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Projection with explicit low-rank adapters (Eq. (1)-(2), Sec. 3.4)   */
/* ------------------------------------------------------------------ */

/* H bf16 [M][d_in]; W bf16 [d_q + 2 d_kv][d_in] (rows of W_Q, W_K, W_V);
 * A bf16 [3r][d_in] (A_Q, A_K, A_V); Bm bf16 [d_q + 2 d_kv][r] (B_Q, B_K,
 * B_V).  For each row h of H and each output row n of projection p:
 *   y[n] = W[n] . h + scale * B[n] . (A_p h),   scale = alpha / r,
 * the explicit adapter branch (r (d_in + d_out) extra MACs per token).
 * Y is fp64 [M][d_q + 2 d_kv]; Ybf16 (optional) is Y rounded once to bf16. */
int orc_project(const uint16_t* Hm, int M, int d_in, const uint16_t* W, int d_q, int d_kv, const uint16_t* A,
                const uint16_t* Bm, int rank, double scale, double* Y, uint16_t* Ybf16)
{
    if (M < 0 || d_in < 1 || d_q < 1 || d_kv < 1 || rank < 0 || !Y || (M > 0 && (!Hm || !W)))
        return ORC_ERR_ARG;
    if (rank > 0 && (!A || !Bm))
        return ORC_ERR_ARG;
    const int N = d_q + 2 * d_kv;
    int nomem = 0;
    /* rows are independent; each thread has its own buffers */
#pragma omp parallel reduction(| : nomem)
    {
    double* h = (double*)malloc(sizeof(double) * (size_t)d_in);
    double* t = (double*)malloc(sizeof(double) * (size_t)(3 * rank + 1));
    if (!h || !t)
        nomem = 1;
#pragma omp for schedule(dynamic, 4)
    for (int m = 0; m < M; ++m) {
        if (!h || !t)
            continue;
        for (int i = 0; i < d_in; ++i)
            h[i] = bf16_to_f32(Hm[(size_t)m * d_in + i]);
        for (int k = 0; k < 3 * rank; ++k) {
            double acc = 0.0;
            for (int i = 0; i < d_in; ++i)
                acc += (double)bf16_to_f32(A[(size_t)k * d_in + i]) * h[i];
            t[k] = acc;
        }
        for (int n = 0; n < N; ++n) {
            double acc = 0.0;
            for (int i = 0; i < d_in; ++i)
                acc += (double)bf16_to_f32(W[(size_t)n * d_in + i]) * h[i];
            if (rank > 0) {
                int p = n < d_q ? 0 : (n < d_q + d_kv ? 1 : 2);
                double lora = 0.0;
                for (int k = 0; k < rank; ++k)
                    lora += (double)bf16_to_f32(Bm[(size_t)n * rank + k]) * t[p * rank + k];
                acc += scale * lora;
            }
            Y[(size_t)m * N + n] = acc;
            if (Ybf16)
                Ybf16[(size_t)m * N + n] = orc_f64_to_bf16(acc);
        }
    }
    free(h);
    free(t);
    }
    return nomem ? ORC_ERR_NOMEM : ORC_OK;
}

/* ------------------------------------------------------------------ */

/* Dense-merge deployment (Sec. 3.4 "Deployment overhead"): the adapter
 * branch folded into the base weights, which leaves the projection shapes
 * unchanged.  For every output row n of projection p (rows of W_Q, then
 * W_K, then W_V) and input channel i:
 *   W'[n][i] = W[n][i] + scale * sum_k B[n][k] A[p r + k][i],
 * accumulated in fp64.  Wd (optional) receives W' in fp64, Wout (optional)
 * W' rounded once to bf16 (nearest, ties to even).  Same argument shapes as
 * orc_project; rank 0 copies W. */
int orc_merge_adapter(const uint16_t* W, int d_in, int d_q, int d_kv, const uint16_t* A, const uint16_t* Bm,
                      int rank, double scale, double* Wd, uint16_t* Wout)
{
    if (d_in < 1 || d_q < 1 || d_kv < 1 || rank < 0 || !W || (!Wd && !Wout))
        return ORC_ERR_ARG;
    if (rank > 0 && (!A || !Bm))
        return ORC_ERR_ARG;
    const int N = d_q + 2 * d_kv;
#pragma omp parallel for schedule(dynamic, 16)
    for (int n = 0; n < N; ++n) {
        const int p = n < d_q ? 0 : (n < d_q + d_kv ? 1 : 2);
        for (int i = 0; i < d_in; ++i) {
            double upd = 0.0;
            for (int k = 0; k < rank; ++k)
                upd += (double)bf16_to_f32(Bm[(size_t)n * rank + k]) *
                       (double)bf16_to_f32(A[((size_t)p * rank + k) * d_in + i]);
            const double w = (double)bf16_to_f32(W[(size_t)n * d_in + i]) + scale * upd;
            if (Wd)
                Wd[(size_t)n * d_in + i] = w;
            if (Wout)
                Wout[(size_t)n * d_in + i] = orc_f64_to_bf16(w);
        }
    }
    return ORC_OK;
}
