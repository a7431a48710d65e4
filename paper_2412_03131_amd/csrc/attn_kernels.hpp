#pragma once
// attn_kernels.hpp -- decode attention over the differentiated paged KV cache
// for gfx950 (DiffKV Eq. (1) of Sec. 2.1, kernel structure of Sec. 6.2).
//
// Work: a table's pages (high pages first, then low pages) are processed by
// one workgroup for all GQ query heads that read them (eight waves up to GQ
// 5, two workgroups per CU; twelve waves, one per CU, above), or by half of a
// sixteen-wave workgroup that takes two tables, a long one and a short one,
// with its waves split by their work (attn_pair, the automatic mode when the
// tables fill the device), or -- in the balanced mode -- every table's pages
// are laid end to end and cut into one equal share per resident workgroup, so
// the spread of table lengths costs nothing; a table that straddles shares is
// merged by the last of them to finish (split tables below).  Inside a
// workgroup each wave of a segment takes every nw-th page, one register
// buffer per wave and the next page staged in LDS: with four (three) waves per
// SIMD the waves hide each other's page loads.  A wave's page IDs arrive as
// one vector per 64 pages and each page is loaded through a buffer resource
// over that page (scalar address, hardware bounds).
//
// Lane mapping inside a wave (64 lanes = 4 rows of 16):
//   key phase    lane = grp*16 + j: token j (and j+16 on 32-token pages),
//                32-dim group grp.  A row holds its group's q as 16 fp16
//                pairs, one per lane, read by the whole row through DPP
//                row_newbcast, and computes sum(q*code) with v_dot2 on codes
//                turned into fp16 denormals (exact, one v_perm or AND per two
//                codes), then s*sum + z*sum(q) (scale and zero factored out of
//                the dot product).  A transposed sum over the four rows
//                (v_permlane16/32_swap) leaves head 4s + r of token j in
//                row r, so the softmax costs one exp2 per (token, head).
//   softmax      online, base 2, with a lazily raised max: the page max (DPP
//                row ops) is only taken when a logit exceeds the running max
//                by more than 8 (weights up to 2^8).
//   value phase  lane owns dims 2*lane, 2*lane+1 (its row's group).  The
//                weights p*s_v of the row's tokens, rounded to fp16, go
//                through LDS (one broadcast read per token pair for all heads)
//                into v_dot2_f32_f16 with two tokens' codes as fp16 denormals;
//                the zero-point term and the weights' rounding error (charged
//                at the centre code) are accumulated per lane and added once.
// The waves' (max, sum, acc) states merge through LDS.
#include <cstddef>
#include <utility>

#include "attn_common.hpp"

namespace dkv {


// Compile-time description of layout LI (formats and segment offsets of its two
// sections, page bytes); the API selects the instantiation from the caller's
// diffkv_layout.
template <int LI>
struct Lay {
    static constexpr KvFmt hi = kLayoutFmts[LI].hi, lo = kLayoutFmts[LI].lo;
    static constexpr SecOffsets ohi = sec_offsets(hi), olo = sec_offsets(lo);
    static constexpr int page_bytes = layout_page_bytes(LI);
    // value rows wider than 16 bytes per lane (8-bit values) need a second load
    static constexpr int nv = layout_wide_values(LI) ? 2 : 1;
};

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

// ---- cross-lane helpers ------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float fmax_sel(float a, float b) { return a > b ? a : b; }

// max over the 16 lanes of each row, result in every lane of the row
__device__ __forceinline__ float row_max16(float x)
{
    x = fmax_sel(x, dpp<0x128>(x));  // row_ror:8
    x = fmax_sel(x, dpp<0x124>(x));  // row_ror:4
    x = fmax_sel(x, dpp<0x122>(x));  // row_ror:2
    x = fmax_sel(x, dpp<0x121>(x));  // row_ror:1
    return x;
}
__device__ __forceinline__ float row_sum16(float x)
{
    x += dpp<0x128>(x);
    x += dpp<0x124>(x);
    x += dpp<0x122>(x);
    x += dpp<0x121>(x);
    return x;
}

// ---- code conversions ---------------------------------------------------------
// Key codes become fp16 *denormals* (bit pattern = code, value = code * 2^-24):
// one v_perm or one AND per two codes, exact, and exact again in
// v_dot2_f32_f16 (its fp16 products are exact in fp32).  The 2^24 is folded
// into the key scale.  Pairs hold dims (d, d+4) of each 8-dim block, the
// pairing the q registers use (v_perm selector kPermSel below).

__device__ __forceinline__ float dot2(half2_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2(a, __builtin_bit_cast(half2_t, b), c, false);
}
// f(integral_constant<int, 0>) ... f(integral_constant<int, N-1>)
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f)
{
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ---- key dot products against DPP-broadcast query pairs ----------------------
// A row holds its group's 16 query pairs one per lane; lane L's pair reaches
// the whole row through DPP row_newbcast:L on src0 of v_dot2c_f32_f16
// (L = 1 .. 15; row_newbcast:0 does not broadcast, so pair 0 is also kept
// whole in every lane).  The compiler cannot see inside asm, so these
// sequences keep the hardware's wait-state rules themselves:
//   - a DPP instruction reads a VGPR at least 2 wait states after a VALU write
//     of it, and 5 after an EXEC write;
//   - a VALU instruction reads the result of a dot instruction at least 3
//     wait states after it, unless it is the same dot opcode reading it as
//     its accumulator.
// The steps are volatile asm (kept in the order written), each forms the next
// code pair one step ahead, and the no-ops below pad the distances where the
// head count does not.  The query registers are written once, before any page.
template <int N>
__device__ __forceinline__ void kwait()
{
    if constexpr (N > 0) asm volatile("s_nop %0" ::"n"(N - 1));
}
template <int L>
__device__ __forceinline__ void kdot_bcast(float& c, uint32_t q, uint32_t x)
{
    static_assert(L >= 1 && L <= 15, "row_newbcast lane");
    asm volatile("v_dot2c_f32_f16_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf" : "+v"(c) : "v"(q), "v"(x), "n"(L));
}
__device__ __forceinline__ void kdot_first(float& c, half2_t q, uint32_t x)
{
    asm volatile("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(c) : "v"(q), "v"(x));
}
__device__ __forceinline__ uint32_t kperm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    uint32_t x;
    asm volatile("v_perm_b32 %0, %1, %2, %3" : "=v"(x) : "v"(hi), "v"(lo), "s"(sel));
    return x;
}
__device__ __forceinline__ uint32_t kand(uint32_t v, uint32_t mask)
{
    uint32_t x;
    asm volatile("v_and_b32 %0, %2, %1" : "=v"(x) : "v"(v), "s"(mask));
    return x;
}
// The next code pair's v_perm / v_and and the first head's dot in one asm
// statement (the compiler pads between separate asm statements).
template <int L>
__device__ __forceinline__ uint32_t kperm_dot(uint32_t hi, uint32_t lo, uint32_t sel, float& c, uint32_t q,
                                              uint32_t x)
{
    uint32_t xn;
    asm volatile("v_perm_b32 %0, %2, %3, %4\n\tv_dot2c_f32_f16_dpp %1, %5, %6 row_newbcast:%7 row_mask:0xf bank_mask:0xf"
                 : "=&v"(xn), "+v"(c)
                 : "v"(hi), "v"(lo), "s"(sel), "v"(q), "v"(x), "n"(L));
    return xn;
}
template <int L>
__device__ __forceinline__ uint32_t kand_dot(uint32_t v, uint32_t mask, float& c, uint32_t q, uint32_t x)
{
    uint32_t xn;
    asm volatile("v_and_b32 %0, %3, %2\n\tv_dot2c_f32_f16_dpp %1, %4, %5 row_newbcast:%6 row_mask:0xf bank_mask:0xf"
                 : "=&v"(xn), "+v"(c)
                 : "v"(v), "s"(mask), "v"(q), "v"(x), "n"(L));
    return xn;
}

constexpr int kMax0(int a) { return a > 0 ? a : 0; }

// End of a sequence: three wait states, then each result passes through an
// empty asm, so no instruction the compiler schedules can read a result before
// the wait (the wait itself only orders against other volatile asm).
template <int GQ>
__device__ __forceinline__ void kdone(float (&d)[GQ])
{
    kwait<3>();
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) asm volatile("" : "+v"(d[hh]));
}

// A query pair times 1/16 (both halves, fp16, rounded to nearest): the
// factor of the K4 pairs whose codes are taken as 16 * code.  Exact unless a
// half falls below 2^-10 in magnitude, where the fp16 denormal spacing rounds
// it by at most 2^-25 (2^-21 of the unscaled value).
__device__ __forceinline__ uint32_t q_by16(uint32_t q)
{
    const half2_t s = {(_Float16)0.0625f, (_Float16)0.0625f};
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2_t, q) * s);
}

// v_perm selector of pair a of an 8-dim block: bytes [w_lo.byte a, 0, w_hi.byte a, 0]
constexpr uint32_t kPermSel(int a) { return 0x0C000C00u | ((uint32_t)(4 + a) << 16) | (uint32_t)a; }

// K8 token: d[h] = sum over the group's 16 pairs of q_h . codes (w = the 32
// code bytes of the token's group).  Step i forms pair i+1 and adds pair i.
// Between the same head's steps i-1 and i lie GQ-1 dots and the next pair's
// v_perm (none in the last step); step 1 follows the first products of
// another dot opcode (3 wait states), later steps the same one (the DPP rule,
// 2).  The code pair of step i was formed before GQ dots of step i-1.
template <int GQ>
__device__ __forceinline__ void kdots_k8(const uint32_t (&w)[8], const uint32_t (&qr)[GQ], const half2_t (&q0)[GQ],
                                         float (&d)[GQ])
{
    kwait<5>();
    uint32_t x = kperm(w[1], w[0], kPermSel(0));
    static_for<16>([&](auto i) {
        constexpr int perm = i < 15 ? 1 : 0;
        constexpr int pad = i > 0 ? kMax0((i == 1 ? 3 : 2) - (GQ - 1 + perm)) : 0;
        constexpr int m1 = (i + 1) / 4, a1 = (i + 1) % 4;
        uint32_t xn = 0;
        if constexpr (i > 0 && i < 15 && pad == 0) {
            // next pair and head 0 in one statement, then the other heads
            xn = kperm_dot<(i > 0 ? i : 1)>(w[2 * m1 + 1], w[2 * m1], kPermSel(a1), d[0], qr[0], x);
#pragma unroll
            for (int hh = 1; hh < GQ; ++hh) kdot_bcast<(i > 0 ? i : 1)>(d[hh], qr[hh], x);
        } else {
            if constexpr (i < 15) xn = kperm(w[2 * m1 + 1], w[2 * m1], kPermSel(a1));
            kwait<pad>();
#pragma unroll
            for (int hh = 0; hh < GQ; ++hh) {
                if constexpr (i == 0) kdot_first(d[hh], q0[hh], x);
                else kdot_bcast<(i > 0 ? i : 1)>(d[hh], qr[hh], x);
            }
        }
        x = xn;
    });
    kdone<GQ>(d);
}

// K4 token: pairs 4m + a (a = 0..3) of dword w[m] are its nibbles (a, a+4)
// (a even) or 16 * nibbles (a, a+4) (a odd: one AND, no shift); odd pairs take
// the query pairs scaled by 1/16 (qr16), so all sixteen pairs sum into one
// chain per head, with the timing of the K8 sequence (an AND in place of each
// v_perm).
template <int GQ>
__device__ __forceinline__ void kdots_k4(const uint32_t (&w)[4], const uint32_t (&qr)[GQ], const uint32_t (&qr16)[GQ],
                                         const half2_t (&q0)[GQ], float (&d)[GQ])
{
    kwait<5>();
    uint32_t w8[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) w8[m] = w[m] >> 8;
    uint32_t x = kand(w[0], 0x000F000Fu);
    static_for<16>([&](auto i) {
        constexpr int step = i < 15 ? 1 : 0;
        constexpr int pad = i > 0 ? kMax0((i == 1 ? 3 : 2) - (GQ - 1 + step)) : 0;
        constexpr int n = i + 1, m = n / 4, a = n % 4;
        constexpr uint32_t mask = (a & 1) ? 0x00F000F0u : 0x000F000Fu;
        const uint32_t(&q)[GQ] = (i % 2) ? qr16 : qr;
        uint32_t xn = 0;
        if constexpr (i > 0 && i < 15 && pad == 0) {
            xn = kand_dot<(i > 0 ? i : 1)>(a >= 2 ? w8[m] : w[m], mask, d[0], q[0], x);
#pragma unroll
            for (int hh = 1; hh < GQ; ++hh) kdot_bcast<(i > 0 ? i : 1)>(d[hh], q[hh], x);
        } else {
            if constexpr (i < 15) xn = kand(a >= 2 ? w8[m] : w[m], mask);
            kwait<pad>();
#pragma unroll
            for (int hh = 0; hh < GQ; ++hh) {
                if constexpr (i == 0) kdot_first(d[hh], q0[hh], x);
                else kdot_bcast<(i > 0 ? i : 1)>(d[hh], q[hh], x);
            }
        }
        x = xn;
    });
    kdone<GQ>(d);
}

constexpr float kTwo24 = 16777216.0f;

// Raw bytes of one page as one lane needs them.  High and low pages take
// the same seven loads (two of them unused on high pages, re-reading lines the
// page's other loads fetch), so one buffer serves both page loops without
// register copies.
struct PageRaw {
    uint4 k0, k1;  // high: K8 chunks 2g, 2g+1 of token j; low: K4 chunk g of tokens j, j+16
    uint4 vr;      // V code rows of dims 2*lane, 2*lane+1 (the first 16 bytes)
    uint4 vr2;     // 8-bit values: the next 16 bytes (the row of dim 2*lane+1)
    uint32_t m0;   // K meta {s, z} of token j, group g
    uint32_t m1;   // low: K meta of token j+16
    uint32_t m2;   // V meta of token j, group g
    uint32_t m3;   // low: V meta of token j+16
};


// One wave's next page, written into LDS by the seven loads themselves (buffer
// loads with an LDS destination: lane L's 16- or 4-byte piece lands at index L
// of its row), so a page can be in flight while the wave computes another one
// from registers without holding a second register buffer.
template <int NV>
struct PageStage {
    uint4 k0[kWave];
    uint4 k1[kWave];
    uint4 vr[NV][kWave];
    uint32_t m[4][kWave];
};

typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) _Float16 lds_f16;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4 lds_u4;
typedef __attribute__((address_space(3))) float lds_f32;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) f32x4 lds_f4;

// Buffer loads with an LDS destination: lane L's 16 (or 4) bytes land at byte
// m0 + 16 L (or m0 + 4 L).  Written as asm so that the compiler, which would
// otherwise make every later LDS access wait for them, leaves their waits to
// take_page (the only reader of the slot).
__device__ __forceinline__ void lds_load16(u32x4 rs, uint32_t m0, uint32_t voff, uint32_t soff)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 ::"s"(m0), "v"(voff), "s"(rs), "s"(soff) : "memory");
}
__device__ __forceinline__ void lds_load4(u32x4 rs, uint32_t m0, uint32_t voff, uint32_t soff)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                 ::"s"(m0), "v"(voff), "s"(rs), "s"(soff) : "memory");
}

// Stage a page of format F (section offsets O) into the wave's slot: through a
// buffer resource over the one page (base pg, the layout's page bytes: the
// hardware bounds every access), with LDS destinations.  Lane (group g, token
// j): the key codes of token j's group (K8: chunks 2g, 2g+1; K4: chunk g of
// tokens j and j + 16), its key metadata (and token j + 16's), the value rows of
// dims 2*lane, 2*lane+1, and the value metadata of group g for tokens j, j + 16.
template <int KB, int VB, int T, int NV>
__device__ __forceinline__ void stage_page(PageStage<NV>& sg, const uint8_t* pg, int pbytes, SecOffsets O, int lane)
{
    const uint32_t grp = (uint32_t)lane >> 4, jl = (uint32_t)lane & 15;
    const unsigned long long base = (unsigned long long)pg;
    const u32x4 rs = {(uint32_t)base, (uint32_t)(base >> 32) & 0xffffu, (uint32_t)pbytes, 0x00020000u};
    const uint32_t kc0 = (uint32_t)O.kc + ((KB == 8 ? 2 * grp : grp) * T + jl) * 16;
    const uint32_t kc1 = KB == 8 ? kc0 + T * 16 : (T == 32 ? kc0 + 256 : kc0);
    const uint32_t km0 = (uint32_t)O.km + jl * 16 + grp * 4;
    const uint32_t km1 = T == 32 ? km0 + 256 : km0;
    constexpr uint32_t rowb = 2 * T * VB / 8;  // bytes of the lane's two value rows
    const uint32_t vc = (uint32_t)O.vc + (uint32_t)lane * rowb;
    const uint32_t vm0 = (uint32_t)O.vm + (grp * T + jl) * 4;
    const uint32_t vm1 = T == 32 ? vm0 + 64 : vm0;
    const uint32_t m0 = (uint32_t)(size_t)(__attribute__((address_space(3))) void*)&sg;
    constexpr uint32_t om = offsetof(PageStage<NV>, m);
    static_assert(offsetof(PageStage<NV>, k1) == 1024 && offsetof(PageStage<NV>, vr) == 2048, "stage slot layout");
    static_assert(NV == 2 || rowb <= 16, "value rows wider than one load");
    lds_load16(rs, m0, kc0, 0u);
    lds_load16(rs, m0 + 1024, kc1, 0u);
    lds_load16(rs, m0 + 2048, vc, 0u);  // rows of 8 bytes per lane: the next lane's share comes along
    if constexpr (NV == 2) lds_load16(rs, m0 + 3072, rowb > 16 ? vc + 16 : vc, 0u);
    lds_load4(rs, m0 + om, km0, 0u);
    lds_load4(rs, m0 + om + 256, km1, 0u);
    lds_load4(rs, m0 + om + 512, vm0, 0u);
    lds_load4(rs, m0 + om + 768, vm1, 0u);
}

// The staged page into registers: wait for the wave's staging loads (every
// vector load of the wave, the only ones in flight here being the slot's),
// read the slot, and wait for the reads, so the next staging loads cannot
// overwrite the slot before it is read.
template <int NV>
__device__ __forceinline__ void take_page(PageRaw& r, const PageStage<NV>& sg, int lane)
{
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    r.k0 = sg.k0[lane];
    r.k1 = sg.k1[lane];
    r.vr = sg.vr[0][lane];
    if constexpr (NV == 2) r.vr2 = sg.vr[NV - 1][lane];
    r.m0 = sg.m[0][lane];
    r.m1 = sg.m[1][lane];
    r.m2 = sg.m[2][lane];
    r.m3 = sg.m[3][lane];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

template <int GQ>
struct WaveState {
    static constexpr int NS = (GQ + 3) / 4;  // head slots per lane in the softmax layout
    float m[NS];       // running max of head 4s + row (log2 domain), row-uniform
    float mt[NS];      // m + kSlack: the raise threshold on pages that take the slack
    float l[NS];       // this lane's share of the running sum of head 4s + row
    float z[GQ];       // this lane's share of the zero-point term of head hh (group = row)
    float acc[GQ][2];  // dims 2*lane, 2*lane+1, in units of 2^-24
};

// LDS for the value weights of one page: [row = value group][token pair][head]
// as fp16 pairs; rows padded by four dwords so the four rows' broadcast reads
// hit different banks.
template <int GQ, int NW>
struct CoefLds {
    static constexpr int kH = GQ <= 4 ? 4 : 8;  // heads per pair entry (dwords)
    static constexpr int kRow = 16 * kH + 4;     // dwords per row (16 pairs)
    uint32_t v[NW][4 * kRow];
};
static_assert(4 * CoefLds<1, 8>::kRow >= 32 * 4, "a wave's weight area holds one slot's softmax weights");

// Sum over the four rows with a transpose: row r of the result holds the sum of
// argument r (heads a, b, c, d -> rows 0, 1, 2, 3).
__device__ __forceinline__ float xsum4(float a, float b, float c, float d)
{
    auto ab = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    auto cd = __builtin_amdgcn_permlane16_swap(__float_as_uint(c), __float_as_uint(d), false, false);
    const float u = __uint_as_float(ab[0]) + __uint_as_float(ab[1]);
    const float w = __uint_as_float(cd[0]) + __uint_as_float(cd[1]);
    auto uw = __builtin_amdgcn_permlane32_swap(__float_as_uint(u), __float_as_uint(w), false, false);
    return __uint_as_float(uw[0]) + __uint_as_float(uw[1]);
}

// Sum over the four rows, in every row (same column).
__device__ __forceinline__ float rows_allsum(float v)
{
    auto ab = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    const float u = __uint_as_float(ab[0]) + __uint_as_float(ab[1]);
    auto uw = __builtin_amdgcn_permlane32_swap(__float_as_uint(u), __float_as_uint(u), false, false);
    return __uint_as_float(uw[0]) + __uint_as_float(uw[1]);
}

// Whether slot s of a wave's GQ heads (heads 4s .. 4s+3, one per row) holds a
// single head: the last slot when GQ = 4k + 1.  Its logit is then summed over
// the rows into every row, so its weights need no gather across rows.
template <int GQ>
constexpr bool lone_slot(int s)
{
    return GQ % 4 == 1 && s == (GQ + 3) / 4 - 1;
}

// The transposed row sum of slot s: row r gets head 4s + r (a lone head: every row).
template <int GQ>
__device__ __forceinline__ float slot_sum(int s, const float* part)
{
    return lone_slot<GQ>(s) ? rows_allsum(part[4 * s])
                            : xsum4(part[4 * s], part[4 * s + 1], part[4 * s + 2], part[4 * s + 3]);
}

// o[r] = x of row r (same column), in every lane
__device__ __forceinline__ void gather4(float x, float* o)
{
    auto eo = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    auto e = __builtin_amdgcn_permlane32_swap(eo[0], eo[0], false, false);
    auto od = __builtin_amdgcn_permlane32_swap(eo[1], eo[1], false, false);
    o[0] = __uint_as_float(e[0]);
    o[1] = __uint_as_float(od[0]);
    o[2] = __uint_as_float(e[1]);
    o[3] = __uint_as_float(od[1]);
}

// Softmax weights are exp2(logit - m) with a running max m that is only
// raised when a logit exceeds it by more than kSlack (weights stay <= 2^8),
// on pages whose V scales are at most 2^7 (fp16 bits 0x5800; scales are never
// negative, so the bit pattern orders them); other pages raise it to their max.
constexpr float kSlack = 8.0f;
constexpr uint32_t kVScaleSlackMax = 0x5800u;

// One page: logits, online softmax, weighted value sum.  NT = tokens per lane.
//
// Value weights.  For token j, head h and value group g the weight
// w = p * s_v is rounded to fp16 (c) and multiplied with the codes on
// v_dot2_f32_f16 (codes as fp16 denormals, products exact in fp32).  The
// rounding error (w - c) is charged to the zero-point term at the centre code
// ((2^bits - 1)/2): sum_j p*z_v + centre*(w - c), so what is left of it scales
// with |code - centre| <= half the code range, at most 2^-12 of the group's
// value range per unit of softmax weight.  2-bit codes in odd crumbs are
// extracted as 4*code, and their c carries w/4.
//
// Page format (KB, VB, T): K8 pages hold 16 tokens (one per lane), K4 pages 16
// or 32 (NT = T/16 tokens per lane).  Value token pairs per format, token t of
// the page: V4/16 nibbles (t, t+4) of a dword; V2/32 and V2/16 crumbs (t, t+8);
// V8/16 bytes (2i, 2i+1); V1/32 bits (t, t+16).
template <int VB, int T>
__device__ __forceinline__ void coef_slot(int t, int& pi, int& pos)
{
    if constexpr (VB == 4 && T == 16) { pi = (t >> 3) * 4 + (t & 3); pos = (t >> 2) & 1; }
    else if constexpr (VB == 2 && T == 32) { pi = (t >> 4) * 8 + (t & 7); pos = (t >> 3) & 1; }
    else if constexpr (VB == 2 && T == 16) { pi = t & 7; pos = t >> 3; }
    else if constexpr (VB == 8 && T == 16) { pi = t >> 1; pos = t & 1; }
    else { static_assert(VB == 1 && T == 32, "page format"); pi = t & 15; pos = t >> 4; }
}

template <int GQ, int KB, int VB, int T>
__device__ __forceinline__ void do_page(WaveState<GQ>& st, const PageRaw& r, const uint32_t (&qr)[GQ],
                                        const uint32_t (&qr16)[GQ], const half2_t (&q0)[GQ],
                                        const float (&qs2)[GQ], float sl2, int n_valid, int lane,
                                        lds_u32* coef_row, lds_f32* px)
{
    constexpr int NS = WaveState<GQ>::NS;
    constexpr int kH = CoefLds<GQ, 8>::kH;
    constexpr int NT = T / 16;
    static_assert(KB == 4 || NT == 1, "8-bit keys: 16 tokens per page");
    const int jl = lane & 15;
    // ---- logits: lane (group row, token jl) partial dot products, then a
    // transposed row sum: afterwards row r holds head 4s + r of token jl + 16*tk
    float lg[NT][NS];
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        const uint32_t km = tk ? r.m1 : r.m0;
        // the zero term takes the fp16 zero as it is (a mixed-precision fma),
        // qs2 = sum(q) * scale_log2 per head
        const float ks = h2f(km & 0xffffu) * (kTwo24 * sl2);
        const float kz = (float)__builtin_bit_cast(f16x2, km).y;
        float dk[GQ];
        if constexpr (KB == 8) {
            const uint32_t w[8] = {r.k0.x, r.k0.y, r.k0.z, r.k0.w, r.k1.x, r.k1.y, r.k1.z, r.k1.w};
            kdots_k8<GQ>(w, qr, q0, dk);
        } else {
            const uint4 kk = tk ? r.k1 : r.k0;
            const uint32_t w[4] = {kk.x, kk.y, kk.z, kk.w};
            kdots_k4<GQ>(w, qr, qr16, q0, dk);
        }
        float part[4 * NS];
#pragma unroll
        for (int hh = 0; hh < 4 * NS; ++hh) {
            if (hh < GQ) {
                part[hh] = fmaf(kz, qs2[hh], ks * dk[hh]);
            } else {
                part[hh] = 0.f;
            }
        }
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            if (lone_slot<GQ>(s)) {
                // a lone head's row sum through the wave's exchange area: one
                // write, one read and three adds instead of two copies, two
                // swaps and two adds (same order: (r0 + r1) + (r2 + r3))
                px[(jl + 16 * tk) * 4 + (lane >> 4)] = part[4 * s];
                const f32x4 v = *reinterpret_cast<const lds_f4*>(px + (jl + 16 * tk) * 4);
                lg[tk][s] = (v.x + v.y) + (v.z + v.w);
            } else {
                lg[tk][s] = slot_sum<GQ>(s, part);
            }
        }
    }
    // tokens past the section's end (only on its last page: a uniform branch,
    // kept a branch by the empty asm, which the compiler does not speculate)
    if (n_valid < T) {
        asm volatile("");
#pragma unroll
        for (int tk = 0; tk < NT; ++tk)
#pragma unroll
            for (int s = 0; s < NS; ++s)
                if (jl + 16 * tk >= n_valid) lg[tk][s] = -INFINITY;
    }
    // ---- online softmax with a lazily raised max (one head per lane and slot).
    // The value weights p * s_v are rounded to fp16, so they must stay below
    // 65504: on a page whose V scales all lie at or below 2^7 the slack keeps
    // p <= 2^8 (weights <= 2^15); a page with a larger V scale takes no slack,
    // so its weights are p <= 1 times an fp16 scale.
    const bool big_v = (r.m2 & 0xffffu) > kVScaleSlackMax || (NT == 2 && (r.m3 & 0xffffu) > kVScaleSlackMax);
    // one wave-wide compare mask per logit, or-ed on the scalar unit
    unsigned long long raise = 0;
    if (__builtin_amdgcn_ballot_w64(big_v)) {
        asm volatile("");
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int tk = 0; tk < NT; ++tk) raise |= __builtin_amdgcn_ballot_w64(lg[tk][s] > st.m[s]);
    } else {
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int tk = 0; tk < NT; ++tk) raise |= __builtin_amdgcn_ballot_w64(lg[tk][s] > st.mt[s]);
    }
    if (raise) {
        float al[4 * NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            float mx = lg[0][s];
            if (NT > 1) mx = fmax_sel(mx, lg[NT - 1][s]);
            mx = row_max16(mx);
            const float mnew = fmax_sel(st.m[s], mx);
            const float alpha = __builtin_amdgcn_exp2f(st.m[s] - mnew);
            st.m[s] = mnew;
            st.mt[s] = mnew + kSlack;
            st.l[s] *= alpha;
            if (lone_slot<GQ>(s))
                al[4 * s] = alpha;
            else
                gather4(alpha, al + 4 * s);
        }
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            st.z[hh] *= al[hh];
            st.acc[hh][0] *= al[hh];
            st.acc[hh][1] *= al[hh];
        }
    }
    float p[NT][NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) {
            p[tk][s] = __builtin_amdgcn_exp2f(lg[tk][s] - st.m[s]);
            st.l[s] += p[tk][s];
        }
    }
    // ---- value weights of token jl + 16*tk for this lane's group (row), all
    // heads: fp16 to LDS, zero-point and rounding terms into z.  First every
    // slot's heads (one per row) of the lane's tokens reach every row through
    // LDS: a write and a read on the LDS pipe instead of three lane swaps and
    // their copies on the VALU (the wave's LDS operations complete in order, so
    // a read sees all four rows).  The exchange uses the start of the wave's
    // weight area, so all of it ends before the first weight is written there.
    float pg[NT][4 * NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (lone_slot<GQ>(s)) {
#pragma unroll
            for (int tk = 0; tk < NT; ++tk) pg[tk][4 * s] = p[tk][s];
            continue;
        }
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) px[(jl + 16 * tk) * 4 + (lane >> 4)] = p[tk][s];
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) {
            const f32x4 v = *reinterpret_cast<const lds_f4*>(px + (jl + 16 * tk) * 4);
            pg[tk][4 * s] = v.x;
            pg[tk][4 * s + 1] = v.y;
            pg[tk][4 * s + 2] = v.z;
            pg[tk][4 * s + 3] = v.w;
        }
    }
    lds_f16* crow = reinterpret_cast<lds_f16*>(coef_row);
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        const uint32_t vm = tk ? r.m3 : r.m2;
        const float vs = h2f(vm & 0xffffu), vz = h2f(vm >> 16);
        constexpr float centre = 0.5f * (float)((1 << VB) - 1);
        const int tok = jl + 16 * tk;
        const bool by4 = VB == 2 && (tok & 1);
        // s_v times the lane's code factor (2-bit values) in one mixed-precision fma
        const float vs_c = VB == 2 ? fmaf(vs, by4 ? 0.25f : 1.0f, 0.0f) : vs;
        const float cc = by4 ? 4.f * centre : centre;
        const float zc = fmaf(centre, vs, vz);
        int pi, pos;
        coef_slot<VB, T>(tok, pi, pos);
        lds_f16* dst = crow + pi * 2 * kH + pos;
        // weights rounded to fp16 two heads at a time (one packed conversion);
        // the second of a pair goes to LDS straight from the high half
        // (ds_write_b16_d16_hi: the wave's LDS operations stay in order, and
        // the asm orders itself against the compiler's memory accesses)
        _Float16 c[GQ];
        uint32_t cpk[(GQ + 1) / 2];
#pragma unroll
        for (int hh = 0; hh < GQ; hh += 2) {
            if (hh + 1 < GQ) {
                const f32x2 w2 = {pg[tk][hh] * vs_c, pg[tk][hh + 1] * vs_c};
                const f16x2 c2 = __builtin_convertvector(w2, f16x2);
                c[hh] = c2.x;
                c[hh + 1] = c2.y;
                cpk[hh / 2] = __builtin_bit_cast(uint32_t, c2);
            } else {
                c[hh] = (_Float16)(pg[tk][hh] * vs_c);
            }
        }
        const uint32_t dst_addr = (uint32_t)(size_t)dst;
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            st.z[hh] = fmaf(pg[tk][hh], zc, st.z[hh]);
            st.z[hh] = fmaf(-cc, (float)c[hh], st.z[hh]);
            if (hh % 2 == 1)
                asm volatile("ds_write_b16_d16_hi %0, %1 offset:%2" ::"v"(dst_addr), "v"(cpk[hh / 2]), "i"(4 * hh) : "memory");
            else
                dst[2 * hh] = c[hh];
        }
    }
    __builtin_amdgcn_wave_barrier();
    // ---- value phase: lane owns dims 2*lane, 2*lane+1 (its row's group); token
    // pairs of each dword as fp16 denormals, one v_dot2 per pair and head.
    const uint32_t w[4] = {r.vr.x, r.vr.y, r.vr.z, r.vr.w};
    // weights of token pairs p0 .. p0+3, all heads (four broadcast reads per
    // pair group, issued together)
    auto read_cf = [&](int p0, half2_t (&cf)[4][GQ]) {
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {
            const lds_u32* src = coef_row + (p0 + pp) * kH;
            uint32_t t[kH];
#pragma unroll
            for (int i = 0; i < kH; i += 4) {
                const u32x4 v = *reinterpret_cast<const lds_u4*>(src + i);
                t[i] = v.x; t[i + 1] = v.y; t[i + 2] = v.z; t[i + 3] = v.w;
            }
#pragma unroll
            for (int hh = 0; hh < GQ; ++hh) cf[pp][hh] = __builtin_bit_cast(half2_t, t[hh]);
        }
    };
    auto dots = [&](const half2_t (&cf)[GQ], uint32_t xa, uint32_t xb) {
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            st.acc[hh][0] = dot2(cf[hh], xa, st.acc[hh][0]);
            st.acc[hh][1] = dot2(cf[hh], xb, st.acc[hh][1]);
        }
    };
    if constexpr (VB == 4 && T == 16) {
        // 16 tokens x 4 bits per 64-bit row; nibbles k, k+4 of dword dw -> pair 4*dw + k
#pragma unroll
        for (int dw = 0; dw < 2; ++dw) {
            half2_t cf[4][GQ];
            read_cf(4 * dw, cf);
            const uint32_t a = w[dw], b = w[2 + dw];
#pragma unroll
            for (int k = 0; k < 4; ++k) dots(cf[k], (a >> (4 * k)) & 0x000F000Fu, (b >> (4 * k)) & 0x000F000Fu);
        }
    } else if constexpr (VB == 2) {
        // 2-bit rows of T tokens; dword `half` of a row holds tokens 16*half + r
        // at bits 2r; crumbs r, r+8 -> pair 8*half + (r & 7) (4*code for odd r)
        constexpr int halves = T / 16;
#pragma unroll
        for (int half = 0; half < halves; ++half) {
            const uint32_t a = T == 32 ? w[half] : w[0], b = T == 32 ? w[2 + half] : w[1];
#pragma unroll
            for (int q4 = 0; q4 < 2; ++q4) {
                half2_t cf[4][GQ];
                read_cf(8 * half + 4 * q4, cf);
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    const int s4 = 2 * q4 + s2;
                    const uint32_t ya = a >> (4 * s4), yb = b >> (4 * s4);
                    dots(cf[2 * s2], ya & 0x00030003u, yb & 0x00030003u);
                    dots(cf[2 * s2 + 1], ya & 0x000C000Cu, yb & 0x000C000Cu);
                }
            }
        }
    } else if constexpr (VB == 8) {
        // 16 tokens x 8 bits per 128-bit row (dims 2*lane: vr, 2*lane + 1: vr2);
        // bytes 2i, 2i+1 of the row -> pair i
        const uint32_t wb[4] = {r.vr2.x, r.vr2.y, r.vr2.z, r.vr2.w};
#pragma unroll
        for (int q4 = 0; q4 < 2; ++q4) {
            half2_t cf[4][GQ];
            read_cf(4 * q4, cf);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int i2 = 4 * q4 + k, m = i2 >> 1;
                const uint32_t sel = (i2 & 1) ? 0x0C030C02u : 0x0C010C00u;
                dots(cf[k], __builtin_amdgcn_perm(w[m], w[m], sel), __builtin_amdgcn_perm(wb[m], wb[m], sel));
            }
        }
    } else {
        // 32 tokens x 1 bit per 32-bit row; bits r, r+16 -> pair r
        const uint32_t a = w[0], b = w[1];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            half2_t cf[4][GQ];
            read_cf(4 * q4, cf);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int rr = 4 * q4 + k;
                dots(cf[k], (a >> rr) & 0x00010001u, (b >> rr) & 0x00010001u);
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------------------
// Tables and their work
// ---------------------------------------------------------------------------
// A table's pages in attention order: high pages 0 .. ph-1 (slots 0 ..), then
// low pages ph .. np-1 (slots p_max-1 downward).  For balancing, a high page
// is kHighUnits units of work and a low page kLowUnits: the page loops are
// bound by VALU issue, and a 32-token low page issues twice the instructions
// of a 16-token high page (both bytes per page being equal), a 16-token low
// page about as many.  A table's first page also carries `seg` units, the
// cost of starting a segment (its query, page-ID and first-page loads, the
// waves' merge, an arrival), so a balanced share that crosses a table boundary
// gets fewer pages: page 0 starts at unit 0, page p > 0 at seg + hi*p
// (p <= ph) or seg + hi*ph + lo*(p - ph).  Ranking tables by work and
// splitting a paired workgroup's waves count a table's start as `seg_pair`
// units instead (each measured best for its own use: the balanced shares with
// 50, the pairs with 80).
template <int LI>
struct Units {
    static constexpr int hi = 3;
    static constexpr int lo = Lay<LI>::lo.T == 32 ? 6 : 3;
    static constexpr int seg = 50;
    static constexpr int seg_pair = 80;
};

struct TableInfo {
    int ph, np;
    int len_hi, len_lo;
    long long units;
};

template <int LI>
__device__ __forceinline__ TableInfo table_info_of(const AttnArgs& a, int len_hi, int len_lo)
{
    constexpr int kHighUnits = Units<LI>::hi, kLowUnits = Units<LI>::lo;
    constexpr int kTh = Lay<LI>::hi.T, kTl = Lay<LI>::lo.T;
    TableInfo ti;
    const int P = a.p_max;
    ti.len_hi = len_hi;
    ti.len_lo = len_lo;
    // page counts from the section lengths, clamped to the table width
    int ph = (ti.len_hi + kTh - 1) / kTh;
    int pl = (ti.len_lo + kTl - 1) / kTl;
    ph = ph < 0 ? 0 : (ph > P ? P : ph);
    pl = pl < 0 ? 0 : (pl > P - ph ? P - ph : pl);
    ti.ph = ph;
    ti.np = ph + pl;
    ti.units = ti.np > 0 ? Units<LI>::seg + (long long)kHighUnits * ph + (long long)kLowUnits * pl : 0;
    return ti;
}
// A table's work as ranking and pairing count it (start cost seg_pair).
template <int LI>
__device__ __forceinline__ long long pair_units(const TableInfo& ti)
{
    return ti.np > 0 ? ti.units - Units<LI>::seg + Units<LI>::seg_pair : 0;
}
// t uniform: the section lengths come through scalar loads (the attention
// kernels never write them), so everything derived from them stays scalar.
template <int LI>
__device__ __forceinline__ TableInfo table_info(const AttnArgs& a, int t)
{
    const auto* len = (const __attribute__((address_space(4))) int32_t*)(a.len + 2 * (long long)t);
    return table_info_of<LI>(a, len[0], len[1]);
}

// first page whose first unit is >= x (np if none)
template <int LI>
__device__ __forceinline__ int page_at_unit(long long x, int ph, int np)
{
    constexpr int kHighUnits = Units<LI>::hi, kLowUnits = Units<LI>::lo;
    if (x <= 0) return 0;
    x -= Units<LI>::seg;
    if (x <= 0) return np > 0 ? 1 : 0;
    const long long xh = (long long)kHighUnits * ph;
    const long long p = x <= xh ? (x + kHighUnits - 1) / kHighUnits : ph + (x - xh + kLowUnits - 1) / kLowUnits;
    return p > np ? np : (int)p;
}

template <int GQ, int NW>
struct AttnShared {
    float m[NW][8];
    float l[NW][8];
    float acc[NW][GQ][kD];
    long long scan[NW + 1];
    int t_first;
    long long u_first;
    int rk_t[2];       // tables of the ranks searched (longest-first ranking)
    int rk_len[2][2];  // and their section lengths
    int last;          // this workgroup is the last of a split table's shares
    unsigned long long tag;  // this call's tag (arrival words)
    long long units;         // balanced mode: the unit total of all tables
    int pend_t[2];           // balanced mode: split tables of this share, and
    long long pend_u[2];     // their first units (arrivals after the walk)
};

// Exclusive prefix sum of one 64-bit value per thread of an NW-wave workgroup.
template <int NW>
__device__ __forceinline__ long long wg_excl_scan(long long x, long long* lds, long long* total)
{
    const int l = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
    long long inc = x;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const long long y = __shfl_up(inc, o, kWave);
        if (l >= o) inc += y;
    }
    if (l == kWave - 1) lds[w] = inc;
    __syncthreads();
    long long before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const long long v = lds[i];
        before += i < w ? v : 0;
        tot += v;
    }
    __syncthreads();
    *total = tot;
    return before + inc - x;
}

__device__ __forceinline__ void write_empty(const AttnArgs& a, int t, int gq)
{
    const int b = t / a.Hkv, h = t - b * a.Hkv;
    for (int i = threadIdx.x; i < gq * kD; i += blockDim.x) {
        const int hh = i / kD, d = i - hh * kD;
        const long long row = (long long)b * a.Hq + h * gq + hh;
        a.out[row * kD + d] = 0.f;
        if (d == 0 && a.lse) a.lse[row] = -INFINITY;
    }
}

// The same from one thread (an empty table met by one thread of the balanced
// mode's table scan).
__device__ __forceinline__ void write_empty_one(const AttnArgs& a, int t, int gq)
{
    const int b = t / a.Hkv, h = t - b * a.Hkv;
    for (int hh = 0; hh < gq; ++hh) {
        const long long row = (long long)b * a.Hq + h * gq + hh;
        float4* o = reinterpret_cast<float4*>(a.out + row * kD);
        for (int i = 0; i < kD / 4; ++i) o[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (a.lse) a.lse[row] = -INFINITY;
    }
}

// ---- split tables: merged by the last of their shares -------------------
// A table whose pages went to n > 1 workgroups is merged inside the launch
// by the last of them to finish.  Each writes its partial state {max, sum,
// acc} per head with agent-scope stores (written through to memory, where
// every XCD's accesses meet), waits until they are done, and counts itself in
// the table's arrival word with agent-scope atomics; the one that brings the
// count to n reads the n states back with agent-scope loads, in page order,
// and writes the output.  Every byte that crosses workgroups goes through
// agent-scope accesses, so no cache-wide release or acquire (an L2 writeback
// and invalidate per workgroup) is needed.
//
// The arrival words (call_tag, arrive_count) count at most 65535 split ranges
// or the share count plus one per table.

__device__ __forceinline__ void put_part(float* p, float v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 get_part2(const float* p)  // p 8-byte aligned
{
    const unsigned long long v = __hip_atomic_load(reinterpret_cast<unsigned long long*>(const_cast<float*>(p)),
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

// The kernel's arguments read afresh from the kernel argument segment (the
// attention kernel's one argument sits at its start), through a pointer the
// compiler cannot see through: what the code after the page loops reads from
// it is loaded there, not at the kernel's start and kept in registers across
// the loops.
__device__ __forceinline__ const AttnArgs& late_args()
{
    typedef const __attribute__((address_space(4))) AttnArgs* karg_ptr;
    karg_ptr p = (karg_ptr)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(p));
    return *(const AttnArgs*)p;
}

// After the workgroup wrote its partial state of table t: whether it is the
// n-th of the table's shares to arrive (uniform over the workgroup).
template <int GQ, int NW>
__device__ __forceinline__ bool arrive_last(const AttnArgs& a, AttnShared<GQ, NW>& sh, int t, int n)
{
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's partial stores are done
    __syncthreads();
    if (threadIdx.x == 0) sh.last = arrive_count(a.arrive + t, sh.tag) == (unsigned long long)n;
    __syncthreads();
    return __builtin_amdgcn_readfirstlane(sh.last) != 0;
}

// Output of table t from the partial states of its nsl share slots at `base`
// (slot j at base + j * GQ * kPartStride; wrote(j): slot j holds a state), in
// page order.  One wave per query head, lane = dims 2*lane, 2*lane+1; the
// first kPre slots' loads are all issued before any is used (one round trip
// for the usual two to five shares of a table).
template <int GQ, typename Wrote>
__device__ __forceinline__ void merge_parts(const AttnArgs& a, int t, const float* base, int nsl, Wrote wrote)
{
    const int b = t / a.Hkv, h = t - b * a.Hkv;
    const int lane = threadIdx.x & (kWave - 1);
    const int hh = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const long long stride = (long long)GQ * kPartStride;
    static_assert(GQ <= 8, "one wave per query head (eight or more waves)");
    if (hh < GQ) {
        const float* pr = base + hh * kPartStride;
        constexpr int kPre = 8;
        float2 ml[kPre], o[kPre];
#pragma unroll
        for (int j = 0; j < kPre; ++j) {
            const bool ok = j < nsl && wrote(j);
            ml[j] = ok ? get_part2(pr + j * stride) : make_float2(-INFINITY, 0.f);
            o[j] = ok ? get_part2(pr + j * stride + 2 + 2 * lane) : make_float2(0.f, 0.f);
        }
        float M = -INFINITY;
#pragma unroll
        for (int j = 0; j < kPre; ++j) M = fmax_sel(M, ml[j].x);
        for (int j = kPre; j < nsl; ++j)
            if (wrote(j)) M = fmax_sel(M, get_part2(pr + j * stride).x);
        float L = 0.f, O0 = 0.f, O1 = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int j = 0; j < kPre; ++j) {
                const float f = __builtin_amdgcn_exp2f(ml[j].x - M);  // 0 for slots without a state
                L = fmaf(ml[j].y, f, L);
                O0 = fmaf(o[j].x, f, O0);
                O1 = fmaf(o[j].y, f, O1);
            }
            for (int j = kPre; j < nsl; ++j) {
                if (!wrote(j)) continue;
                const float2 mj = get_part2(pr + j * stride), oj = get_part2(pr + j * stride + 2 + 2 * lane);
                const float f = __builtin_amdgcn_exp2f(mj.x - M);
                L = fmaf(mj.y, f, L);
                O0 = fmaf(oj.x, f, O0);
                O1 = fmaf(oj.y, f, O1);
            }
        }
        const long long row = (long long)b * a.Hq + h * GQ + hh;
        *reinterpret_cast<float2*>(a.out + row * kD + 2 * lane) =
            (L > 0.f) ? make_float2(O0 / L, O1 / L) : make_float2(0.f, 0.f);
        if (lane == 0 && a.lse) a.lse[row] = (L > 0.f) ? (M + __log2f(L)) * 0.69314718055994530942f : -INFINITY;
    }
    __syncthreads();  // sh.last is read again by the next arrival
}

// ---------------------------------------------------------------------------
// One segment: pages [pa, pb) of table t for all GQ query heads of its KV
// head, taken by waves w0 .. w0+nw-1 of the workgroup: wave w0 + i takes every
// nw-th page from pa + i, each loading a page and then computing it (the other
// waves on its SIMD cover the wait).  seg_pages leaves each wave's (max, sum,
// acc) state in LDS (no workgroup barrier inside, so the waves of a workgroup
// may work on different tables); seg_merge combines the states of waves
// w0 .. w0+nw-1 into the output (part == nullptr) or into a partial state
// {max, sum, acc} per head at `part` (pa == pb gives the empty state).
// ---------------------------------------------------------------------------
template <int GQ, int LI, int NW>
__device__ __forceinline__ void seg_pages(const AttnArgs& a, AttnShared<GQ, NW>& sh, CoefLds<GQ, NW>* coef,
                                          PageStage<Lay<LI>::nv>* stage, int t, const TableInfo& ti, int pa,
                                          int pb, int w0, int nw, int& done, int target)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wv = wave - w0;  // this wave's place among the segment's waves
    const int grp = lane >> 4;
    const int P = a.p_max;
    const int b = t / a.Hkv, h = t - b * a.Hkv;
    const int ph = ti.ph;
    const float sl2 = a.scale_log2;
    const long long npool = a.num_pages;
    using LY = Lay<LI>;
    constexpr long long page_bytes = LY::page_bytes;  // (the layout check guarantees it)
    lds_u32* coef_row = (lds_u32*)(&coef->v[wave][grp * CoefLds<GQ, NW>::kRow]);
    // one slot's softmax weights [token][row] pass through the start of the wave's
    // weight area before the page's weights are written there
    lds_f32* px = (lds_f32*)(&coef->v[wave][0]);
    const int nmine = pb - pa > wv ? (pb - pa - wv + nw - 1) / nw : 0;
    const int32_t* trow = a.page_table + (long long)t * P;

    // The wave's pages run in chunks of 64: lane k holds the ID of chunk page
    // c0 + k (one vector load per chunk), and a page's ID is read into a scalar
    // register when its loads are issued.  Chunk bounds [c0, c1); past c1 the
    // index is clamped to the chunk's last page.
    auto page_of = [&](int i) { return pa + wv + nw * i; };
    auto slot_of = [&](int p) { return p < ph ? p : P - 1 - (p - ph); };
    int c0 = 0, c1 = 0, c_last = 0, ids_v = 0;
    auto clamp_i = [&](int i) { return i < c_last ? i : c_last; };
    auto load_ids = [&]() {
        const int k = c0 + lane;
        return trow[slot_of(page_of(clamp_i(k)))];
    };
    // Stage page i in this wave's LDS slot; ok = page i exists and lies in the
    // pool.  The loads are unconditional (an index past the chunk's last page
    // re-reads it; an ID outside the pool reads page 0 and is not computed).
    PageStage<LY::nv>& sg = stage[wave];
    const uint32_t npool32 = npool > 0x7fffffffLL ? 0x80000000u : (uint32_t)npool;
    auto issue = [&](int i, bool& ok) {
        const int ic = clamp_i(i);
        const int id = __builtin_amdgcn_readlane(ids_v, ic - c0);
        const bool in_pool = (uint32_t)id < npool32;  // never read outside the pool
        ok = i < c1 && in_pool;
        const uint8_t* pg = a.pool + (in_pool ? id : 0) * page_bytes;
        if (page_of(ic) < ph) stage_page<LY::hi.kb, LY::hi.vb, LY::hi.T, LY::nv>(sg, pg, (int)page_bytes, LY::ohi, lane);
        else stage_page<LY::lo.kb, LY::lo.vb, LY::lo.T, LY::nv>(sg, pg, (int)page_bytes, LY::olo, lane);
    };
    // The query loads go first: they depend only on the table, so their
    // latency overlaps the page-ID -> page chain below.  Lane k of a row loads
    // the two dwords of its pair k (dims 8(k/4) + k%4 and +4: dwords x, z or
    // y, w of the 8-dim block) and the two of pair 0.
    const int qm = (lane & 15) >> 2, qa = lane & 3;
    uint32_t qraw[GQ][4];
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const uint32_t* qd = reinterpret_cast<const uint32_t*>(a.q + ((long long)b * a.Hq + h * GQ + hh) * kD + grp * kG);
        const int o = 4 * qm + ((qa & 2) ? 1 : 0);
        qraw[hh][0] = qd[o];
        qraw[hh][1] = qd[o + 2];
        qraw[hh][2] = qd[0];
        qraw[hh][3] = qd[2];
    }

    PageRaw buf0;
    bool ok0 = false, ok_next = false;
    // first chunk: its IDs and first page go out beside the query loads
    c1 = nmine < kWave ? nmine : kWave;
    c_last = c1 > 0 ? c1 - 1 : 0;
    if (nmine > 0) {
        ids_v = load_ids();
        issue(0, ok_next);
    }

    // q of this lane's group as fp16 pairs (d, d+4), one pair per lane (read
    // by the others through DPP), pair 0 (dims 0, 4) in every lane; qs2 = the
    // group's sum (row sum) times scale_log2
    uint32_t qr[GQ], qr16[GQ];
    half2_t q0[GQ];
    float qs2[GQ];
    constexpr uint32_t kOnes = 0x3C003C00u;  // fp16 pair (1, 1)
    {
        const uint32_t sel = (qa & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            qr[hh] = __builtin_amdgcn_perm(qraw[hh][1], qraw[hh][0], sel);
            qr16[hh] = q_by16(qr[hh]);
            q0[hh] = __builtin_bit_cast(half2_t, __builtin_amdgcn_perm(qraw[hh][3], qraw[hh][2], 0x05040100u));
            qs2[hh] = row_sum16(dot2(__builtin_bit_cast(half2_t, qr[hh]), kOnes, 0.f)) * sl2;
        }
    }

    WaveState<GQ> st;
#pragma unroll
    for (int s = 0; s < WaveState<GQ>::NS; ++s) {
        st.m[s] = -INFINITY;
        st.mt[s] = -INFINITY;
        st.l[s] = 0.f;
    }
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        st.z[hh] = 0.f;
        st.acc[hh][0] = st.acc[hh][1] = 0.f;
    }

    // This wave's pages i < nhi are high pages, the rest low pages.  High and
    // low pages run in loops of their own (no per-page branch between two
    // different updates of the softmax state); the prefetch crosses from one
    // loop to the next.
    const int nhi = ph - pa - wv > 0 ? min(nmine, (ph - pa - wv + nw - 1) / nw) : 0;
    auto compute_hi = [&](int i, const PageRaw& r, bool ok) {
        if (i >= c1 || !ok) return;
        const int p = page_of(i);
        do_page<GQ, LY::hi.kb, LY::hi.vb, LY::hi.T>(st, r, qr, qr16, q0, qs2, sl2, ti.len_hi - p * LY::hi.T, lane, coef_row,
                                                   px);
    };
    auto compute_lo = [&](int i, const PageRaw& r, bool ok) {
        if (i >= c1 || !ok) return;
        const int p = page_of(i);
        do_page<GQ, LY::lo.kb, LY::lo.vb, LY::lo.T>(st, r, qr, qr16, q0, qs2, sl2, ti.len_lo - (p - ph) * LY::lo.T, lane,
                                                   coef_row, px);
    };
    // Wave priority.  One workgroup per table or range (target 0): it follows
    // the pages this wave still has, so on a SIMD shared with shorter work the
    // longest work is served first (longest-first scheduling at the wave
    // level).  Balanced shares (equal work, target = the wave's part of its
    // share in units): it follows the part still ahead of the wave, falling
    // at 60, 30 and 10 % left, so whichever of the waves on a SIMD is further
    // behind goes first and the two workgroups of a CU finish together; with
    // one level for all, issue goes to the older wave, and the workgroup
    // dispatched first ran ahead while its partner finished alone, two waves
    // per SIMD.  `done` counts the units of the wave's pages taken so far.
    auto set_prio = [&](int rem, int units) {
        if (target > 0) {
            const int left = target - done;
            if (left * 10 > target * 6) __builtin_amdgcn_s_setprio(3);
            else if (left * 10 > target * 3) __builtin_amdgcn_s_setprio(2);
            else if (left * 10 > target) __builtin_amdgcn_s_setprio(1);
            else __builtin_amdgcn_s_setprio(0);
            done += units;
        } else {
            if (rem > 12) __builtin_amdgcn_s_setprio(3);
            else if (rem > 6) __builtin_amdgcn_s_setprio(2);
            else if (rem > 2) __builtin_amdgcn_s_setprio(1);
            else __builtin_amdgcn_s_setprio(0);
        }
    };
    // Page i comes out of the LDS slot into registers, page i + 1 goes into the
    // slot, then page i is computed: one page is always in flight while the
    // wave computes.
    auto next = [&](int i) {
        take_page(buf0, sg, lane);
        ok0 = ok_next;
        if (i + 1 < c1) issue(i + 1, ok_next);
    };
    while (c0 < nmine) {
        const int nh = nhi < c1 ? nhi : c1;  // high pages end (within this chunk)
        int i = c0;
        for (; i < nh; ++i) {
            set_prio(nmine - i, Units<LI>::hi);
            next(i);
            compute_hi(i, buf0, ok0);
        }
        for (; i < c1; ++i) {
            set_prio(nmine - i, Units<LI>::lo);
            next(i);
            compute_lo(i, buf0, ok0);
        }
        // next chunk (tables longer than 64 pages per wave): its IDs, then its
        // first page
        c0 = c1;
        c1 = nmine - c0 < kWave ? nmine : c0 + kWave;
        c_last = c1 > c0 ? c1 - 1 : c0;
        if (c0 < nmine) {
            ids_v = load_ids();
            issue(c0, ok_next);
        }
    }

    // ---- finish the wave: row sums of l (head 4s + row) and of the
    // zero-point term (head hh, group = row); acc back from units of 2^-24
#pragma unroll
    for (int s = 0; s < WaveState<GQ>::NS; ++s) {
        const float l = row_sum16(st.l[s]);
        if ((lane & 15) == 0 && 4 * s + grp < GQ) {
            sh.m[wave][4 * s + grp] = st.m[s];
            sh.l[wave][4 * s + grp] = l;
        }
    }
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const float z = row_sum16(st.z[hh]);
        sh.acc[wave][hh][2 * lane] = fmaf(st.acc[hh][0], kTwo24, z);
        sh.acc[wave][hh][2 * lane + 1] = fmaf(st.acc[hh][1], kTwo24, z);
    }
}

template <int GQ, int NW>
__device__ __forceinline__ void seg_merge(const AttnArgs& a, AttnShared<GQ, NW>& sh, int t, int w0, int nw,
                                          float* part)
{
    // ---- merge the waves: final output, or this segment's partial state ---
    const int b = t / a.Hkv, h = t - b * a.Hkv;
    for (int i = threadIdx.x; i < GQ * kD; i += NW * kWave) {
        const int hh = i / kD, d = i - hh * kD;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            if (w >= w0 && w < w0 + nw) M = fmax_sel(M, sh.m[w][hh]);
        float L = 0.f, O = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                if (w < w0 || w >= w0 + nw) continue;
                const float f = __builtin_amdgcn_exp2f(sh.m[w][hh] - M);
                L = fmaf(sh.l[w][hh], f, L);
                O = fmaf(sh.acc[w][hh][d], f, O);
            }
        }
        if (part == nullptr) {
            const long long row = (long long)b * a.Hq + h * GQ + hh;
            a.out[row * kD + d] = (L > 0.f) ? O / L : 0.f;
            if (d == 0 && a.lse) a.lse[row] = (L > 0.f) ? (M + __log2f(L)) * 0.69314718055994530942f : -INFINITY;
        } else {
            float* pr = part + hh * kPartStride;
            put_part(pr + 2 + d, O);
            if (d == 0) {
                put_part(pr, M);
                put_part(pr + 1, L);
            }
        }
    }
}

// One segment by all waves of the workgroup: the pages, then the merge.
template <int GQ, int LI, int NW = attn_waves(GQ, LI)>
__device__ __forceinline__ void run_segment(const AttnArgs& a, AttnShared<GQ, NW>& sh, CoefLds<GQ, NW>* coef,
                                            PageStage<Lay<LI>::nv>* stage, int t, const TableInfo& ti, int pa,
                                            int pb, float* part, int& done, int target)
{
    seg_pages<GQ, LI, NW>(a, sh, coef, stage, t, ti, pa, pb, 0, NW, done, target);
    __syncthreads();
    seg_merge<GQ, NW>(a, sh, t, 0, NW, part);
    __syncthreads();  // LDS is reused by the next segment
}

// ---------------------------------------------------------------------------
// attn_decode.
//  splits = S >= 1: workgroup t*S + c takes range c of table t's pages, cut
//    into min(S, pages) equal ranges (S = 1: no split).
//  splits = 0: balanced shares.  All tables' pages, in table order, form one
//    list of U work units; workgroup k of W owns the pages whose first unit
//    lies in [k*U/W, (k+1)*U/W).  Each workgroup finds its first table with a
//    prefix sum over the tables' units, then walks its tables.  A table lying
//    inside one share is finished in place; otherwise share k writes its
//    partial state to slot k + t (distinct for every (share, table) pair met
//    in this walk) and the last of the table's shares to arrive merges them.
//    An empty table's output is written by workgroup t % W.
// ---------------------------------------------------------------------------
// Tables of ranks rank[0 .. NR) when the tables are ordered by decreasing
// work units (bucketed into 1024 bins, ties by index): workgroups are
// dispatched in index order and two share a CU for the whole launch, so
// taking the tables longest first spreads the long ones over the CUs and
// starts them first (longest-processing-time-first order).  Every workgroup
// derives the same order from the section lengths; wave 0 does it alone
// (wave-level scans, no workgroup barrier until the result).  Beyond kRankPer
// tables per lane the order is the identity.  ti[k] gets the table's pages and
// units, from the lengths the ranking wave already holds.
constexpr int kKeep = 8;     // tables per thread whose units stay in registers (balanced mode)
constexpr int kRankPer = 16;  // tables per lane of the ranking wave

template <int GQ, int LI, int NW, int NR>
__device__ __forceinline__ void rank_tables(const AttnArgs& a, AttnShared<GQ, NW>& sh, CoefLds<GQ, NW>* coef, int T,
                                            const int (&rank)[NR], int (&tab)[NR], TableInfo (&ti)[NR])
{
    static_assert(NR <= 2, "two ranks at most");
    constexpr int kBins = 1024;
    const int per = (T + kWave - 1) / kWave;
    if (per > kRankPer) {
#pragma unroll
        for (int k = 0; k < NR; ++k) {
            tab[k] = rank[k];
            ti[k] = table_info<LI>(a, rank[k]);
        }
        return;
    }
    static_assert(sizeof(CoefLds<GQ, NW>) >= kBins * sizeof(int), "histogram lives in the weight LDS");
    if (threadIdx.x < kWave) {
        int* hist = reinterpret_cast<int*>(coef);  // free until the page loop
        const int lane = threadIdx.x;
        const int t0 = lane * per, t1 = t0 + per < T ? t0 + per : T;
        int shift = 0;
        while (((Units<LI>::lo * a.p_max + Units<LI>::seg_pair) >> shift) >= kBins) ++shift;
        int lh[kRankPer], ll[kRankPer], bin[kRankPer];
#pragma unroll
        for (int i = 0; i < kRankPer; ++i) {
            const int tc = t0 + i < T ? t0 + i : T - 1;
            lh[i] = i < per ? a.len[2 * tc] : 0;
            ll[i] = i < per ? a.len[2 * tc + 1] : 0;
        }
        static_assert(kBins == 16 * kWave, "sixteen bins per lane");
#pragma unroll
        for (int q = 0; q < 16; q += 4) *reinterpret_cast<int4*>(hist + 16 * lane + q) = make_int4(0, 0, 0, 0);
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < kRankPer; ++i) {
            bin[i] = -1;
            if (t0 + i < t1) {
                const long long u = pair_units<LI>(table_info_of<LI>(a, lh[i], ll[i])) >> shift;
                bin[i] = kBins - 1 - (int)(u < kBins - 1 ? u : kBins - 1);  // bin 0 holds the longest
                atomicAdd(&hist[bin[i]], 1);
            }
        }
        wave_lds_sync();
        int c16[16], s16 = 0;
#pragma unroll
        for (int q = 0; q < 16; q += 4) {
            const int4 v = *reinterpret_cast<const int4*>(hist + 16 * lane + q);
            c16[q] = v.x; c16[q + 1] = v.y; c16[q + 2] = v.z; c16[q + 3] = v.w;
        }
#pragma unroll
        for (int q = 0; q < 16; ++q) s16 += c16[q];
        const int incl = wave_incl_scan(s16);
#pragma unroll
        for (int k = 0; k < NR; ++k) {
            const int j = rank[k];
            int at = incl - s16, b = 0, r = 0;
            bool found = false;
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                if (!found && at <= j && j < at + c16[q]) {
                    found = true;
                    b = 16 * lane + q;
                    r = j - at;
                }
                at += c16[q];
            }
            const unsigned long long fm = __builtin_amdgcn_ballot_w64(found);  // exactly one lane (j < T)
            const int src = fm ? __builtin_ctzll(fm) : 0;
            b = __builtin_amdgcn_readlane(b, src);
            r = __builtin_amdgcn_readlane(r, src);
            // the r-th table (by index) of bin b
            int cnt = 0;
#pragma unroll
            for (int i = 0; i < kRankPer; ++i) cnt += bin[i] == b;
            int before = wave_incl_scan(cnt) - cnt, t = 0, th = 0, tl = 0;
            found = false;
#pragma unroll
            for (int i = 0; i < kRankPer; ++i) {
                if (bin[i] == b) {
                    if (before == r) {
                        found = true;
                        t = t0 + i;
                        th = lh[i];
                        tl = ll[i];
                    }
                    ++before;
                }
            }
            const unsigned long long fm2 = __builtin_amdgcn_ballot_w64(found);
            const int src2 = fm2 ? __builtin_ctzll(fm2) : 0;
            // read with every lane active
            const int tr = __builtin_amdgcn_readlane(t, src2);
            const int thr = __builtin_amdgcn_readlane(th, src2), tlr = __builtin_amdgcn_readlane(tl, src2);
            if (lane == 0) {
                sh.rk_t[k] = tr;
                sh.rk_len[k][0] = thr;
                sh.rk_len[k][1] = tlr;
            }
        }
    }
    __syncthreads();
    // (uniform values read back from LDS: readfirstlane keeps the tables'
    // loads and addresses scalar)
#pragma unroll
    for (int k = 0; k < NR; ++k) {
        ti[k] = table_info_of<LI>(a, __builtin_amdgcn_readfirstlane(sh.rk_len[k][0]),
                                  __builtin_amdgcn_readfirstlane(sh.rk_len[k][1]));
        tab[k] = __builtin_amdgcn_readfirstlane(sh.rk_t[k]);
    }
}

// The table of rank j (see rank_tables).
template <int GQ, int LI, int NW>
__device__ __forceinline__ int longest_first(const AttnArgs& a, AttnShared<GQ, NW>& sh, CoefLds<GQ, NW>* coef, int T, int j,
                                             TableInfo* ti)
{
    const int rank[1] = {j};
    int tab[1];
    TableInfo tis[1];
    rank_tables<GQ, LI, NW, 1>(a, sh, coef, T, rank, tab, tis);
    *ti = tis[0];
    return tab[0];
}

template <int GQ, int LI>
__global__ __launch_bounds__(attn_waves(GQ, LI) * kWave, attn_blocks_per_cu(GQ, LI)) void attn_decode(AttnArgs a)
{
    constexpr int NW = attn_waves(GQ, LI);
    constexpr int NT = NW * kWave;
    __shared__ AttnShared<GQ, NW> sh;
    __shared__ CoefLds<GQ, NW> coef;
    __shared__ PageStage<Lay<LI>::nv> stage[NW];
    // the call tag goes to LDS at once, so the registers it comes in are free
    // for the rest of the kernel (read after the workgroup's first barrier)
    if (threadIdx.x == 0) sh.tag = call_tag();
    const int T = a.B * a.Hkv;
    if (a.splits > 0) {
        const int j = blockIdx.x / a.splits, c = blockIdx.x - j * a.splits;
        TableInfo ti;
        const int t = longest_first<GQ, LI>(a, sh, &coef, T, j, &ti);
        const int n = ti.np < a.splits ? ti.np : a.splits;
        if (n == 0) {
            if (c == 0) write_empty(a, t, GQ);
            return;
        }
        if (c >= n) return;
        const int pa = (int)((long long)c * ti.np / n), pb = (int)((long long)(c + 1) * ti.np / n);
        float* base = a.part + (long long)t * a.splits * GQ * kPartStride;
        float* part = n == 1 ? nullptr : base + (long long)c * GQ * kPartStride;
        int done = 0;
        run_segment<GQ, LI>(a, sh, &coef, stage, t, ti, pa, pb, part, done, 0);
        if (part != nullptr) {
            const AttnArgs& al = late_args();
            if (arrive_last<GQ>(al, sh, t, n)) merge_parts<GQ>(al, t, base, n, [](int) { return true; });
        }
        return;
    }
    // ---- balanced shares -------------------------------------------------
    const long long k = blockIdx.x, W = gridDim.x;
    const int per = (T + NT - 1) / NT;
    const int t0 = threadIdx.x * per;
    const int t1 = t0 + per < T ? t0 + per : T;
    long long units[kKeep];
    long long mine = 0;
    {
        // all loads first (clamped to a valid table), then the units
        int lh[kKeep], ll[kKeep];
#pragma unroll
        for (int i = 0; i < kKeep; ++i) {
            const int tc = t0 + i < T ? t0 + i : T - 1;
            lh[i] = a.len[2 * tc];
            ll[i] = a.len[2 * tc + 1];
        }
#pragma unroll
        for (int i = 0; i < kKeep; ++i) {
            units[i] = t0 + i < t1 ? table_info_of<LI>(a, lh[i], ll[i]).units : 0;
            mine += units[i];
            // an empty table's output comes from workgroup t % W
            if (t0 + i < t1 && units[i] == 0 && (t0 + i) % W == k) write_empty_one(a, t0 + i, GQ);
        }
    }
    for (int t = t0 + kKeep; t < t1; ++t) {
        const long long u = table_info<LI>(a, t).units;
        mine += u;
        if (u == 0 && t % W == k) write_empty_one(a, t, GQ);
    }
    long long total;
    const long long before = wg_excl_scan<NW>(mine, sh.scan, &total);
    if (threadIdx.x == 0) sh.units = total;  // read back by the arrival (not kept in registers)
    const long long b_lo = k * total / W, b_hi = (k + 1) * total / W;
    if (b_lo >= b_hi) return;
    long long u = before;
    for (int t = t0; t < t1; ++t) {  // exactly one table holds unit b_lo
        const int i = t - t0;
        long long n = 0;
#pragma unroll
        for (int j = 0; j < kKeep; ++j) n = i == j ? units[j] : n;
        if (i >= kKeep) n = table_info<LI>(a, t).units;
        if (u <= b_lo && b_lo < u + n) {
            sh.t_first = t;
            sh.u_first = u;
        }
        u += n;
    }
    __syncthreads();
    int t = __builtin_amdgcn_readfirstlane(sh.t_first);
    long long ut = read_lane<long long>(sh.u_first, 0);
    // A share holds at most two split tables, its first and its last (the
    // tables between lie inside it); their arrivals wait until the walk is
    // done, which delays no merge, since the shares end together, and keeps
    // the merge code out of the walk's registers.
    int npend = 0;
    int done = 0;
    const int target = (int)((b_hi - b_lo + NW - 1) / NW);
    while (t < T && ut < b_hi) {
        const TableInfo ti = table_info<LI>(a, t);
        if (ti.units > 0) {
            const int pa = page_at_unit<LI>(b_lo - ut, ti.ph, ti.np);
            const int pb = page_at_unit<LI>(b_hi - ut, ti.ph, ti.np);
            const bool whole = ut >= b_lo && ut + ti.units <= b_hi;
            run_segment<GQ, LI>(a, sh, &coef, stage, t, ti, pa, pb, whole ? nullptr : a.part + (k + t) * GQ * kPartStride,
                                done, target);
            if (!whole) {
                if (threadIdx.x == 0) {
                    sh.pend_t[npend] = t;
                    sh.pend_u[npend] = ut;
                }
                ++npend;
            }
        }
        ut += ti.units;
        ++t;
    }
    const AttnArgs& al = late_args();
    for (int i = 0; i < npend; ++i) {
        __syncthreads();
        const int tp = __builtin_amdgcn_readfirstlane(sh.pend_t[i]);
        const long long up = read_lane<long long>(sh.pend_u[i], 0);
        const long long U = read_lane<long long>(sh.units, 0);
        const long long units = table_info<LI>(al, tp).units;
        // shares kf .. kl own the table's units (the owner of unit x is the
        // largest k with k*U/W <= x); with fewer units than shares some of
        // them own none and wrote nothing
        const long long kf = ((up + 1) * W - 1) / U, kl = ((up + units) * W - 1) / U;
        const int nsl = (int)(kl - kf + 1);
        auto wrote = [&](int j) { return U >= W || (kf + j) * U / W != (kf + j + 1) * U / W; };
        int n = nsl;
        if (U < W) {
            n = 0;
            for (int j = 0; j < nsl; ++j) n += wrote(j) ? 1 : 0;
        }
        if (arrive_last<GQ>(al, sh, tp, n)) merge_parts<GQ>(al, tp, al.part + (kf + tp) * GQ * kPartStride, nsl, wrote);
    }
}

// ---------------------------------------------------------------------------
// attn_pair: the automatic mode when the tables alone fill the device (up to
// GQ 5).  Workgroup j of ceil(T/2), sixteen waves and the whole CU, takes the
// tables of ranks j and T-1-j by decreasing work: a long table with a short
// one, so every CU carries about the average work.  The waves are split
// between the two tables in proportion to their units and take the progress
// priority of the balanced mode, so both tables end together; a long table
// is not left with half a CU once its partner is done, as with one eight-wave
// workgroup per table.  No partial states: each table is finished in place.
// ---------------------------------------------------------------------------
template <int GQ, int LI>
__global__ __launch_bounds__(kPairWaves * kWave, 1) void attn_pair(AttnArgs a)
{
    constexpr int NW = kPairWaves;
    __shared__ AttnShared<GQ, NW> sh;
    __shared__ CoefLds<GQ, NW> coef;
    __shared__ PageStage<Lay<LI>::nv> stage[NW];
    const int T = a.B * a.Hkv;
    const int rank[2] = {(int)blockIdx.x, T - 1 - (int)blockIdx.x};
    int tab[2];
    TableInfo ti[2];
    rank_tables<GQ, LI, NW, 2>(a, sh, &coef, T, rank, tab, ti);
    const bool two = rank[1] != rank[0];
    const long long u0 = pair_units<LI>(ti[0]), u1 = two ? pair_units<LI>(ti[1]) : 0;
    // waves of the first table: of the two integer splits around NW * u0 /
    // (u0 + u1), the one with the smaller larger load per wave (u / waves), at
    // least one wave each
    int n0 = NW;
    if (two && u1 > 0) {
        int lo = (int)(NW * u0 / (u0 + u1));
        lo = lo < 1 ? 1 : (lo > NW - 1 ? NW - 1 : lo);
        const int hi = lo < NW - 1 ? lo + 1 : lo;
        // max(u0/lo, u1/(NW-lo)) <= max(u0/hi, u1/(NW-hi)), compared exactly by cross-multiplying
        auto worse = [&](int n) {  // larger load of split n, as a fraction num/den
            return u0 * (NW - n) >= u1 * n ? std::make_pair(u0, (long long)n) : std::make_pair(u1, (long long)(NW - n));
        };
        const auto wl = worse(lo), wh = worse(hi);
        n0 = wl.first * wh.second <= wh.first * wl.second ? lo : hi;
    }
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const bool first = wave < n0;
    const int tw = first ? tab[0] : tab[1];
    const TableInfo tiw = first ? ti[0] : ti[1];
    const int w0 = first ? 0 : n0, nw = first ? n0 : NW - n0;
    int done = 0;
    const int target = (int)((pair_units<LI>(tiw) + nw - 1) / nw);
    seg_pages<GQ, LI, NW>(a, sh, &coef, stage, tw, tiw, 0, tiw.np, w0, nw, done, target > 0 ? target : 1);
    __syncthreads();
    seg_merge<GQ, NW>(a, sh, tab[0], 0, n0, nullptr);
    if (two) {
        if (n0 < NW) seg_merge<GQ, NW>(a, sh, tab[1], n0, NW - n0, nullptr);
        else write_empty(a, tab[1], GQ);  // no units
    }
}

// ---------------------------------------------------------------------------
// attn_significance: the significance update of one decode step (Sec. 4).  The
// tokens are independent once the lse is known, so a table's pages are cut into
// runs of kSigPages, one workgroup per (table, run); each of its four waves takes
// every fourth page of the run (workgroups past a table's last page exit).  A page's
// key codes, key metadata, scores and positions are loaded; the logits of the
// table's query heads come out of the key phase of do_page (lane = (group, token),
// a transposed row sum), p = exp2(logit - lse) with the attention call's lse, the
// maximum over the heads is taken across the slots and the four rows, and the
// lane of row 0 owning token j rewrites its score as s + (p_max - s) / (N - pos).
// ---------------------------------------------------------------------------

template <int GQ, int KB, int T>
__device__ __forceinline__ void sig_page(const SigArgs& a, uint8_t* pg, int pbytes, SecOffsets O,
                                         const uint32_t (&qr)[GQ], const uint32_t (&qr16)[GQ], const half2_t (&q0)[GQ],
                                         const float (&qsum)[GQ], const float (&lse2)[(GQ + 3) / 4], int n_valid,
                                         int N, int lane)
{
    constexpr int NS = (GQ + 3) / 4;
    constexpr int NT = T / 16;
    const uint32_t grp = (uint32_t)lane >> 4, jl = (uint32_t)lane & 15;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)pg, 0, pbytes, 0x00020000);
    const uint32_t kc0 = (uint32_t)O.kc + ((KB == 8 ? 2 * grp : grp) * T + jl) * 16;
    const uint32_t kc1 = KB == 8 ? kc0 + T * 16 : (T == 32 ? kc0 + 256 : kc0);
    const uint32_t km = (uint32_t)O.km + jl * 16 + grp * 4;
    const uint32_t os = (uint32_t)O.sc, op = (uint32_t)O.pos;
    const uint4 k0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, kc0, 0, 0));
    const uint4 k1 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, kc1, 0, 0));
    const uint32_t m0 = __builtin_amdgcn_raw_buffer_load_b32(rs, km, 0, 0);
    const uint32_t m1 = __builtin_amdgcn_raw_buffer_load_b32(rs, T == 32 ? km + 256 : km, 0, 0);
    float sc[NT];
    int ps[NT];
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        sc[tk] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, os + 4 * (jl + 16 * tk), 0, 0));
        ps[tk] = (int)__builtin_amdgcn_raw_buffer_load_b32(rs, op + 4 * (jl + 16 * tk), 0, 0);
    }
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        const uint32_t kmt = tk ? m1 : m0;
        const float ks = h2f(kmt & 0xffffu) * (kTwo24 * a.scale_log2);
        const float kz = (float)__builtin_bit_cast(f16x2, kmt).y;
        float dk[GQ];
        if constexpr (KB == 8) {
            const uint32_t w[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
            kdots_k8<GQ>(w, qr, q0, dk);
        } else {
            const uint4 kk = tk ? k1 : k0;
            const uint32_t w[4] = {kk.x, kk.y, kk.z, kk.w};
            kdots_k4<GQ>(w, qr, qr16, q0, dk);
        }
        float part[4 * NS];
#pragma unroll
        for (int hh = 0; hh < 4 * NS; ++hh) {
            if (hh < GQ) {
                part[hh] = fmaf(kz, qsum[hh], ks * dk[hh]);
            } else {
                part[hh] = 0.f;
            }
        }
        // row r of slot s holds head 4s + r; its probability, then the maximum
        // over the slots and the four rows
        float x = 0.f;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const float lg = slot_sum<GQ>(s, part);
            const float pr = 4 * s + (int)grp < GQ ? __builtin_amdgcn_exp2f(lg - lse2[s]) : 0.f;
            x = fmax_sel(x, pr);
        }
        // each swap returns the two halves (rows 0-1 | 2-3, then rows 0, 2 | 1, 3)
        // side by side, so their maximum is the maximum over the pair in every lane
        auto sw32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = fmax_sel(__uint_as_float(sw32[0]), __uint_as_float(sw32[1]));
        auto sw16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = fmax_sel(__uint_as_float(sw16[0]), __uint_as_float(sw16[1]));
        const int j = (int)jl + 16 * tk;
        if (grp == 0 && j < n_valid) {
            const float s0 = sc[tk];
            reinterpret_cast<float*>(pg + os)[j] = s0 + (x - s0) / (float)(N - ps[tk]);
        }
    }
}

template <int GQ, int LI>
__global__ __launch_bounds__(kSigWaves * kWave) void attn_significance(SigArgs a)
{
    using LY = Lay<LI>;
    constexpr int NS = (GQ + 3) / 4;
    const int runs = (a.p_max + kSigPages - 1) / kSigPages;
    const int t = blockIdx.x / runs, run = blockIdx.x - t * runs;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int grp = lane >> 4;
    const int b = t / a.Hkv, h = t - b * a.Hkv;
    const int P = a.p_max;
    const auto* lenp = (const __attribute__((address_space(4))) int32_t*)(a.len + 2 * (long long)t);
    const int len_hi = lenp[0], len_lo = lenp[1];
    const int N = a.seq_len[b];
    const int ph = (len_hi + LY::hi.T - 1) / LY::hi.T, np = ph + (len_lo + LY::lo.T - 1) / LY::lo.T;
    const int p_end = np < (run + 1) * kSigPages ? np : (run + 1) * kSigPages;
    if (run * kSigPages >= np) return;
    // q pairs as in run_segment: lane k of a row holds its group's pair k
    // (dims d, d+4), pair 0 whole in every lane, the group's sum
    const int qm = (lane & 15) >> 2, qa = lane & 3;
    uint32_t qr[GQ], qr16[GQ];
    half2_t q0[GQ];
    float qsum[GQ];
    constexpr uint32_t kOnes = 0x3C003C00u;
    const uint32_t sel = (qa & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const uint32_t* qd = reinterpret_cast<const uint32_t*>(a.q + ((long long)b * a.Hq + h * GQ + hh) * kD + grp * kG);
        const int o = 4 * qm + ((qa & 2) ? 1 : 0);
        qr[hh] = __builtin_amdgcn_perm(qd[o + 2], qd[o], sel);
        qr16[hh] = q_by16(qr[hh]);
        q0[hh] = __builtin_bit_cast(half2_t, __builtin_amdgcn_perm(qd[2], qd[0], 0x05040100u));
        qsum[hh] = row_sum16(dot2(__builtin_bit_cast(half2_t, qr[hh]), kOnes, 0.f)) * a.scale_log2;  // times scale_log2
    }
    float lse2[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int hs = 4 * s + grp;
        lse2[s] = hs < GQ ? a.lse[(long long)b * a.Hq + h * GQ + hs] * 1.4426950408889634f : 0.f;
    }
    const int32_t* trow = a.page_table + (long long)t * P;
    for (int p = run * kSigPages + wave; p < p_end; p += kSigWaves) {
        const int id = __builtin_amdgcn_readfirstlane(p < ph ? trow[p] : trow[P - 1 - (p - ph)]);
        if ((unsigned long long)(unsigned)id >= (unsigned long long)a.num_pages) continue;  // never outside the pool
        uint8_t* pg = a.pool + (long long)id * LY::page_bytes;
        if (p < ph)
            sig_page<GQ, LY::hi.kb, LY::hi.T>(a, pg, LY::page_bytes, LY::ohi, qr, qr16, q0, qsum, lse2, len_hi - p * LY::hi.T, N,
                                             lane);
        else
            sig_page<GQ, LY::lo.kb, LY::lo.T>(a, pg, LY::page_bytes, LY::olo, qr, qr16, q0, qsum, lse2,
                                             len_lo - (p - ph) * LY::lo.T, N, lane);
    }
}


// Kernel entry points of layout LI (host-side stubs): which = 0 attn_decode,
// 1 attn_significance, 2 attn_pair (nullptr above GQ 5).
template <int LI>
const void* attn_kernel_of(int gq, int which)
{
#define DKV_ATTN_CASE(G)                                                                   \
    case G:                                                                                \
        if (which == 2) return G <= kPairMaxGq ? reinterpret_cast<const void*>(&attn_pair<(G <= kPairMaxGq ? G : 1), LI>) : nullptr; \
        return which == 0 ? reinterpret_cast<const void*>(&attn_decode<G, LI>)             \
                          : reinterpret_cast<const void*>(&attn_significance<G, LI>);
    switch (gq) {
        DKV_ATTN_CASE(1)
        DKV_ATTN_CASE(2)
        DKV_ATTN_CASE(3)
        DKV_ATTN_CASE(4)
        DKV_ATTN_CASE(5)
        DKV_ATTN_CASE(6)
        DKV_ATTN_CASE(7)
        DKV_ATTN_CASE(8)
    default: return nullptr;
    }
#undef DKV_ATTN_CASE
}

}  // namespace dkv
