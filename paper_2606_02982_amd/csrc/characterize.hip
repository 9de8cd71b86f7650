// Stage 1: whitespace-proxy word counts over a packed UTF-8 prompt buffer.
//
// counts[i] = number of maximal runs of non-whitespace characters in prompt
// i, whitespace being the 29 code points str.split() separates on
// (Sec. "Workload Characterization and Token Budget Estimation").
//
// Byte formulation used here: byte p of prompt i is a word start when p is
// not whitespace and either p is the prompt's first byte or byte p-1 is
// whitespace. A byte is whitespace when it is one of the ASCII separators
// 09-0D, 1C-20, or belongs to one of the multi-byte separators
// C2 85, C2 A0, E1 9A 80, E2 80 80..8A, E2 80 A8, E2 80 A9, E2 80 AF,
// E2 81 9F, E3 80 80 lying entirely inside the prompt. Because none of these
// sequences starts with a continuation byte, this equals decoding each prompt
// on its own (undecodable bytes as ordinary characters) and splitting.
//
// Layout of the work: the text is cut into equal byte ranges, one per
// resident wave; each wave streams its range in super-rounds of 4 KiB (four
// 1 KiB rounds of 64 lanes x 16 bytes, all loads issued together) and
// classifies 4 bytes per 32-bit operation (v_lerp_u8 thresholds). Carries
// between lanes move with DPP wave shifts. A super-round takes one of three
// paths:
//   - no prompt boundary: ASCII classification, with the UTF-8 lead bytes
//     listed in LDS and each checked for a multi-byte separator by one lane;
//   - boundaries but no lead byte: ASCII classification, and per boundary a
//     few lane reads and scalar operations give its exact prefix;
//   - otherwise (and at the ends of a wave's range): round by round, with
//     boundary bits per lane and separators checked at each lead byte.
// Word starts are attributed to prompts through prefix sums: each prompt
// boundary receives the number of word starts in its wave's range before it,
// each wave its total; a second kernel forms counts[i] from the two
// boundaries' local prefixes and the totals of the waves between them. No
// atomics; results are exact integers independent of scheduling.
#include "common.h"
#include "kernels.h"
#include "scoremath.h"

namespace ds {
namespace {

constexpr uint32_t kRound = 1024;        // bytes per wave per round
constexpr uint32_t kLoadRounds = 4;      // rounds loaded together
constexpr uint32_t kBlock = 256;         // 4 independent waves per block
// Each wave takes one contiguous range of the buffer. Four ranges per
// resident wave slot: waves that start late (their slot held by an earlier
// wave or by another stream's kernel) leave a short tail, not a long one.
constexpr uint32_t kRangesPerSlot = 4;
constexpr uint32_t kMaxWaves = 32768;
constexpr uint64_t kNone = ~0ull;

// 0x80 in each byte of x that is an ASCII separator 09-0D or 1C-20.
// v_lerp_u8 averages bytes without carries between them: bit 7 of byte k of
// lerp(x, c, 0) is the carry of x_k + c_k, i.e. x_k >= 0x100 - c_k.
__device__ __forceinline__ uint32_t ascii_space_hb(uint32_t x)
{
    const uint32_t ge09 = __builtin_amdgcn_lerp(x, 0xF7F7F7F7u, 0u);
    const uint32_t ge0e = __builtin_amdgcn_lerp(x, 0xF2F2F2F2u, 0u);
    const uint32_t ge1c = __builtin_amdgcn_lerp(x, 0xE4E4E4E4u, 0u);
    const uint32_t ge21 = __builtin_amdgcn_lerp(x, 0xDFDFDFDFu, 0u);
    return ~ge21 & (ge1c | (ge09 & ~ge0e)) & 0x80808080u;
}

// 0x80 in each byte >= 0xC0 (UTF-8 lead bytes of multi-byte sequences).
__device__ __forceinline__ uint32_t lead_hb(uint32_t x) { return x & (x << 1) & 0x80808080u; }

// bits 7, 15, 23, 31 -> bits 0..3
__device__ __forceinline__ uint32_t compact4(uint32_t hb)
{
    return ((hb >> 7) | (hb >> 14) | (hb >> 21) | (hb >> 28)) & 0xFu;
}

__device__ __forceinline__ uint32_t compact16(uint32_t a, uint32_t b, uint32_t c, uint32_t d)
{
    return compact4(a) | (compact4(b) << 4) | (compact4(c) << 8) | (compact4(d) << 12);
}

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// 16 bytes at c (bytes >= B read as 0). The text is streamed once: the
// full-chunk load is marked nontemporal.
__device__ __forceinline__ uint4 load16(const uint8_t *t, uint64_t B, uint64_t c)
{
    if (c + 16 <= B) {
        v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(t + c));
        return make_uint4(v.x, v.y, v.z, v.w);
    }
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 16; k++)
        if (c + k < B) w[k >> 2] |= (uint32_t)t[c + k] << (8 * (k & 3));
    return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ uint32_t load4(const uint8_t *t, uint64_t B, uint64_t c)
{
    if (c + 4 <= B) return *reinterpret_cast<const uint32_t *>(t + c);
    uint32_t w = 0;
#pragma unroll
    for (int k = 0; k < 4; k++)
        if (c + k < B) w |= (uint32_t)t[c + k] << (8 * k);
    return w;
}

__device__ __forceinline__ uint64_t win_load(const uint64_t *off, uint32_t N, uint32_t wb, int lane)
{
    uint64_t i = (uint64_t)wb + (uint64_t)lane;
    return i <= (uint64_t)N ? off[i] : kNone;
}

// First index i in [0, count) with off[i] >= x, or count (wave-cooperative
// 64-ary search; every step is one round of loads).
__device__ uint32_t lower_bound_wave(const uint64_t *off, uint64_t count, uint64_t x, int lane)
{
    uint64_t lo = 0, hi = count;
    while (hi - lo > 64) {
        uint64_t step = (hi - lo + 63) / 64;
        uint64_t idx = lo + (uint64_t)lane * step;
        bool lt = idx < hi && off[idx] < x;
        uint32_t k = (uint32_t)__popcll(__ballot(lt));
        if (k == 0) { hi = lo; break; }
        uint64_t nlo = lo + (uint64_t)(k - 1) * step + 1;
        uint64_t nhi = lo + (uint64_t)k * step;
        lo = nlo;
        hi = nhi < hi ? nhi : hi;
    }
    bool lt = (lo + (uint64_t)lane < hi) && off[lo + lane] < x;
    return (uint32_t)(lo + (uint64_t)__popcll(__ballot(lt)));
}

// Bytes j..j+3 (little-endian) of the 20-byte window d0..d3, dn.
__device__ __forceinline__ uint32_t bytes_at(const uint4 &d, uint32_t dn, uint32_t j)
{
    uint32_t k = j >> 2, s = j & 3u;
    uint32_t lo = k == 0 ? d.x : k == 1 ? d.y : k == 2 ? d.z : d.w;
    uint32_t hi = k == 0 ? d.y : k == 1 ? d.z : k == 2 ? d.w : dn;
    return __builtin_amdgcn_alignbyte(hi, lo, s);
}

struct WaveState {
    uint32_t s_ptr;     // first boundary index not yet consumed
    uint32_t wb;        // boundary index held by lane 0 of win
    uint64_t win;       // offsets[wb + lane] (kNone past the end)
    uint64_t running;   // word starts in [ws_start, current round)
    uint32_t acc;       // per-lane starts of fast rounds not yet in running
    uint32_t ws_prev;   // whitespace bit of the byte before the round
    uint32_t spill;     // separator bits spilling into the round's first bytes
};

struct RangeCtx {
    const uint64_t *off;
    uint32_t N;
    uint64_t ws_start, ws_end;
    uint32_t *ploc;
};

__device__ __forceinline__ void ensure_window(WaveState &st, const RangeCtx &rc, uint32_t s, int lane)
{
    if (s < st.wb || s - st.wb >= 64) {
        st.wb = s;
        st.win = win_load(rc.off, rc.N, s, lane);
    }
}

// bits 0..3 -> bits 7, 15, 23, 31
__device__ __forceinline__ uint32_t expand4(uint32_t n)
{
    return ((n * 0x204081u) & 0x01010101u) << 7;
}

// Length (2 or 3) of the multi-byte separator starting at the low byte of v
// (bytes little-endian), or 0; branch-free.
__device__ __forceinline__ uint32_t mb_space_len_nb(uint32_t v)
{
    const uint32_t v2 = v & 0xFFFFu, v3 = v & 0xFFFFFFu, b2 = (v >> 16) & 0xFFu;
    const bool two = (v2 == 0x85C2u) | (v2 == 0xA0C2u);
    const bool e2 = (v2 == 0x80E2u) & ((b2 - 0x80u <= 0x0Au) | (b2 == 0xA8u) | (b2 == 0xA9u) | (b2 == 0xAFu));
    const bool three = (v3 == 0x809AE1u) | (v3 == 0x9F81E2u) | (v3 == 0x8080E3u) | e2;
    return two ? 2u : (three ? 3u : 0u);
}

// One 1 KiB round of a wave: lane i holds the 16 bytes at c = rb + 16 i.
// Masks keep 0x80 per byte ("hb" form) as in the ASCII classification.
__device__ __forceinline__ void process_round(WaveState &st, const RangeCtx &rc, const uint4 &d,
                                              uint32_t dn_top, uint64_t rb, int lane)
{
    const uint64_t c = rb + 16u * (uint32_t)lane;
    uint32_t h0 = ascii_space_hb(d.x), h1 = ascii_space_hb(d.y);
    uint32_t h2 = ascii_space_hb(d.z), h3 = ascii_space_hb(d.w);
    const uint32_t l0 = lead_hb(d.x), l1 = lead_hb(d.y), l2 = lead_hb(d.z), l3 = lead_hb(d.w);
    const bool anylead = __ballot((l0 | l1 | l2 | l3) != 0) != 0;

    const bool edge = rb < rc.ws_start || rb + kRound > rc.ws_end;
    const uint64_t lim = rb + kRound + 2;
    ensure_window(st, rc, st.s_ptr, lane);
    const uint64_t nb = readlane64(st.win, (int)(st.s_ptr - st.wb));
    const bool bnd = nb < lim;

    if (!edge && !bnd && st.spill == 0 && !anylead) {
        // no prompt boundary, no multi-byte character starts here, every
        // byte counted: whitespace is the ASCII set (continuation bytes of
        // characters begun earlier are never whitespace on their own)
        uint32_t p0 = wave_shr1(h3, st.ws_prev << 31);
        uint32_t s0 = ~h0 & __builtin_amdgcn_alignbyte(h0, p0, 3);
        uint32_t s1 = ~h1 & __builtin_amdgcn_alignbyte(h1, h0, 3);
        uint32_t s2 = ~h2 & __builtin_amdgcn_alignbyte(h2, h1, 3);
        uint32_t s3 = ~h3 & __builtin_amdgcn_alignbyte(h3, h2, 3);
        st.acc += __popc(s0) + __popc(s1) + __popc(s2) + __popc(s3);
        st.ws_prev = readlane32(h3, 63) >> 31;
        return;
    }

    // boundary bits: bit r set if a prompt starts at byte c + r, r in [0, 18)
    uint32_t bd = 0;
    if (bnd) {
        uint32_t s = st.s_ptr;
        while (true) {
            ensure_window(st, rc, s, lane);
            uint32_t kk = s - st.wb;
            uint64_t m = __ballot((uint32_t)lane >= kk && st.win < lim);
            uint64_t mm = m;
            while (mm) {
                int j = __ffsll((unsigned long long)mm) - 1;
                mm &= mm - 1;
                int64_t r = (int64_t)(readlane64(st.win, j) - c);
                if (r >= 0 && r < 18) bd |= 1u << (uint32_t)r;
            }
            if ((m >> 63) & 1ull) { s = st.wb + 64; if (s > rc.N) break; continue; }
            break;
        }
    }

    // multi-byte separators, checked at lead bytes; a separator must lie
    // inside one prompt. cov: bytes covered, bits 16-17 spill to the next lane.
    uint32_t cov = 0;
    if (anylead) {
        uint32_t lead = compact16(l0, l1, l2, l3);
        const uint32_t dn = wave_shl1(d.x, dn_top);
        while (__ballot(lead != 0)) {
            if (lead) {
                uint32_t j = (uint32_t)__ffs(lead) - 1;
                lead &= lead - 1;
                uint32_t L = mb_space_len_nb(bytes_at(d, dn, j));
                uint32_t inner = (bd >> (j + 1)) & ((1u << (L > 0 ? L - 1 : 0)) - 1u);
                if (L && !inner) cov |= ((1u << L) - 1u) << j;
            }
        }
    }
    const uint32_t spill_out = cov >> 16;
    const uint32_t spill_in = wave_shr1(spill_out, st.spill);
    const uint32_t extra = (cov & 0xFFFFu) | spill_in;
    if (__ballot(extra != 0)) {
        h0 |= expand4(extra & 0xFu);
        h1 |= expand4((extra >> 4) & 0xFu);
        h2 |= expand4((extra >> 8) & 0xFu);
        h3 |= expand4((extra >> 12) & 0xFu);
    }
    st.spill = readlane32(spill_out, 63);

    // word starts: not whitespace, and a prompt start or after whitespace
    const uint32_t p0 = wave_shr1(h3, st.ws_prev << 31);
    st.ws_prev = readlane32(h3, 63) >> 31;
    uint32_t s0 = __builtin_amdgcn_alignbyte(h0, p0, 3);
    uint32_t s1 = __builtin_amdgcn_alignbyte(h1, h0, 3);
    uint32_t s2 = __builtin_amdgcn_alignbyte(h2, h1, 3);
    uint32_t s3 = __builtin_amdgcn_alignbyte(h3, h2, 3);
    if (bnd) {
        s0 |= expand4(bd & 0xFu);
        s1 |= expand4((bd >> 4) & 0xFu);
        s2 |= expand4((bd >> 8) & 0xFu);
        s3 |= expand4((bd >> 12) & 0xFu);
    }
    s0 &= ~h0;
    s1 &= ~h1;
    s2 &= ~h2;
    s3 &= ~h3;
    if (edge) {
        int64_t a = (int64_t)rc.ws_start - (int64_t)c;
        int64_t b = (int64_t)rc.ws_end - (int64_t)c;
        a = a < 0 ? 0 : a;
        b = b > 16 ? 16 : b;
        uint32_t valid = b > a ? (((1u << (uint32_t)b) - 1u) & ~((1u << (uint32_t)a) - 1u)) : 0u;
        s0 &= expand4(valid & 0xFu);
        s1 &= expand4((valid >> 4) & 0xFu);
        s2 &= expand4((valid >> 8) & 0xFu);
        s3 &= expand4((valid >> 12) & 0xFu);
    }
    const uint32_t cnt = (uint32_t)(__popc(s0) + __popc(s1) + __popc(s2) + __popc(s3));
    if (!bnd) {
        st.acc += cnt;
        return;
    }
    // boundary round: exact prefix of word starts at every boundary it owns
    st.running += readlane32(wave_incl_scan_dpp(st.acc), 63);
    st.acc = 0;
    const uint32_t incl = wave_incl_scan_dpp(cnt);
    const uint32_t excl = incl - cnt;
    const uint32_t tot = readlane32(incl, 63);
    const uint32_t start = compact16(s0, s1, s2, s3);
    const uint64_t rend = rb + kRound;
    uint32_t s = st.s_ptr;
    while (true) {
        ensure_window(st, rc, s, lane);
        uint32_t kk = s - st.wb;
        bool cons = (uint32_t)lane >= kk && st.win < rend;
        uint64_t m = __ballot(cons);
        uint64_t rel = st.win - rb;
        int src = (int)((rel >> 4) & 63u);
        uint32_t ex = __shfl(excl, src, 64);
        uint32_t sm = __shfl(start, src, 64);
        if (cons && st.win >= rc.ws_start && st.win < rc.ws_end) {
            uint32_t bit = (uint32_t)(rel & 15u);
            rc.ploc[st.wb + (uint32_t)lane] =
                (uint32_t)st.running + ex + (uint32_t)__popc(sm & ((1u << bit) - 1u));
        }
        if ((m >> 63) & 1ull) { s = st.wb + 64; if (s > rc.N) break; continue; }
        s = st.wb + kk + (uint32_t)__popcll(m);
        break;
    }
    st.s_ptr = s;
    st.running += tot;
}

// Per-wave LDS of the super-round path: the super-round's bytes (plus the
// next 16), the list of lead-byte offsets, and separator coverage per
// (lane, round).
constexpr uint32_t kSR = kRound * kLoadRounds;   // 4 KiB
constexpr uint32_t kMaxLeads = 512;              // more leads: per-round path
struct WaveLds {
    uint32_t data[(kSR + 16) / 4];
    uint16_t slot[kMaxLeads];
    uint32_t cov[32 * kLoadRounds];              // [lane pair][round], 16 bits per lane
};

// Interleaved lead bits of one chunk: bit 8i + k <=> byte 4k + i.
__device__ __forceinline__ uint32_t lead_bits(const uint4 &d)
{
    // bit 7 of each byte of lerp(x, 0x40.., 0): byte >= 0xC0
    const uint32_t gx = __builtin_amdgcn_lerp(d.x, 0x40404040u, 0u);
    const uint32_t gy = __builtin_amdgcn_lerp(d.y, 0x40404040u, 0u);
    const uint32_t gz = __builtin_amdgcn_lerp(d.z, 0x40404040u, 0u);
    const uint32_t gw = __builtin_amdgcn_lerp(d.w, 0x40404040u, 0u);
    return ((gx >> 7) & 0x01010101u) | ((gy >> 6) & 0x02020202u) | ((gz >> 5) & 0x04040404u) |
           ((gw >> 4) & 0x08080808u);
}

__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Multi-byte separators of one whole, boundary-free 4 KiB super-round, all
// lanes cooperating: each lead byte is checked by one lane. Returns 0 (and
// changes nothing) if the super-round holds more than kMaxLeads leads;
// otherwise 1 if no separator was found, 2 if cov[u] (per lane: covered bytes
// of its chunk in round u) or spill_next (bytes past the super-round's end)
// were set. M: the lane's interleaved lead bits, two rounds per 32 bits.
__device__ int superround_separators(WaveLds &L, const uint4 (&d)[kLoadRounds], uint32_t tail,
                                     uint64_t M, uint32_t excl, uint32_t total, int lane,
                                     uint32_t (&cov)[kLoadRounds], uint32_t &spill_next)
{
    if (total > kMaxLeads) return 0;
    // stage the bytes (the coverage words are already zero)
#pragma unroll
    for (uint32_t u = 0; u < kLoadRounds; u++)
        *reinterpret_cast<uint4 *>(&L.data[(u * kRound + 16u * (uint32_t)lane) / 4]) = d[u];
    if (lane == 0) *reinterpret_cast<uint4 *>(&L.data[kSR / 4]) = make_uint4(tail, 0u, 0u, 0u);
    // list the leads as (lane, bit of M), the two halves of M one after the
    // other (32-bit steps); the checking lane finds the byte offset
    uint32_t r = excl;
    const uint32_t lb = (uint32_t)lane << 6;
    uint32_t mlo = (uint32_t)M, mhi = (uint32_t)(M >> 32);
    while (__ballot(mlo != 0)) {
        if (mlo) {
            L.slot[r++] = (uint16_t)(lb | ((uint32_t)__ffs(mlo) - 1u));
            mlo &= mlo - 1u;
        }
    }
    while (__ballot(mhi != 0)) {
        if (mhi) {
            L.slot[r++] = (uint16_t)(lb | ((uint32_t)__ffs(mhi) + 31u));
            mhi &= mhi - 1u;
        }
    }
    wave_lds_fence();
    // check them, one per lane per pass
    bool any = false;
    uint32_t sp = 0;
    for (uint32_t base = 0; base < total; base += 64) {
        uint32_t t = base + (uint32_t)lane;
        uint32_t len = 0, pos = 0;
        if (t < total) {
            // bit p of lane l's M: round u, byte off of the lane's 16
            const uint32_t e = L.slot[t], p = e & 63u, q = p & 31u;
            const uint32_t u = ((p >> 5) << 1) | ((q >> 2) & 1u);
            pos = u * kRound + 16u * (e >> 6) + (((q & 3u) << 2) | (q >> 3));
            uint32_t w0 = L.data[pos >> 2], w1 = L.data[(pos >> 2) + 1];
            len = mb_space_len_nb(__builtin_amdgcn_alignbyte(w1, w0, pos & 3u));
        }
        if (__ballot(len != 0)) {
            any = true;
            for (uint32_t i = 0; i < len; i++) {
                uint32_t b = pos + i;
                const uint32_t bl = (b >> 4) & 63u;
                if (b < kSR) atomicOr(&L.cov[4u * (bl >> 1) + (b >> 10)], 1u << ((b & 15u) + 16u * (bl & 1u)));
                else sp |= 1u << (b - kSR);
            }
        }
    }
    if (!any) return 1;
    spill_next = (__ballot(sp & 1u) ? 1u : 0u) | (__ballot(sp & 2u) ? 2u : 0u);
    wave_lds_fence();
    const uint4 c4 = *reinterpret_cast<const uint4 *>(&L.cov[4 * (lane >> 1)]);
    const uint32_t hs = 16u * ((uint32_t)lane & 1u);
    wave_lds_fence();
    // the coverage words are zero whenever this function starts
    *reinterpret_cast<uint4 *>(&L.cov[4 * (lane >> 1)]) = make_uint4(0u, 0u, 0u, 0u);
    cov[0] = (c4.x >> hs) & 0xFFFFu;
    cov[1] = (c4.y >> hs) & 0xFFFFu;
    cov[2] = (c4.z >> hs) & 0xFFFFu;
    cov[3] = (c4.w >> hs) & 0xFFFFu;
    return 2;
}

// Non-zero if any byte of the lane's 64 bytes has bit 7 set (not ASCII).
__device__ __forceinline__ uint32_t high_any(const uint4 (&d)[kLoadRounds])
{
    uint32_t a = 0;
#pragma unroll
    for (uint32_t u = 0; u < kLoadRounds; u++) a |= d[u].x | d[u].y | d[u].z | d[u].w;
    return a & 0x80808080u;
}

// A whole super-round with no UTF-8 lead byte that holds prompt boundaries
// (the window lanes in bm, in position order). Word starts are those of the
// plain path plus, at a boundary P whose bytes P and P-1 are both
// non-whitespace, the start that the first character of a prompt always is.
// Each boundary receives the exact number of starts in the wave's range
// before it; per boundary only scalar work and lane reads.
__device__ void boundary_superround(WaveState &st, const RangeCtx &rc, const uint4 (&d)[kLoadRounds],
                                    uint64_t sb, uint64_t bm, int lane)
{
    uint64_t base = st.running + readlane32(wave_incl_scan_dpp(st.acc), 63);
    st.acc = 0;
    uint32_t carry = st.ws_prev;
    uint64_t rem = bm;
    uint32_t plv = 0;
    // the boundaries' offsets in the super-round (window lanes in bm: < 4 KiB)
    const uint32_t wrel = (uint32_t)(st.win - sb);
#pragma unroll
    for (uint32_t u = 0; u < kLoadRounds; u++) {
        const uint32_t h0 = ascii_space_hb(d[u].x), h1 = ascii_space_hb(d[u].y);
        const uint32_t h2 = ascii_space_hb(d[u].z), h3 = ascii_space_hb(d[u].w);
        // whitespace bits of each byte's predecessor
        const uint32_t v0 = __builtin_amdgcn_alignbyte(h0, wave_shr1(h3, carry << 31), 3);
        const uint32_t v1 = __builtin_amdgcn_alignbyte(h1, h0, 3);
        const uint32_t v2 = __builtin_amdgcn_alignbyte(h2, h1, 3);
        const uint32_t v3 = __builtin_amdgcn_alignbyte(h3, h2, 3);
        const uint32_t s0 = ~h0 & v0, s1 = ~h1 & v1, s2 = ~h2 & v2, s3 = ~h3 & v3;
        const uint32_t c0 = (uint32_t)__popc(s0), c01 = c0 + (uint32_t)__popc(s1);
        const uint32_t c012 = c01 + (uint32_t)__popc(s2), c = c012 + (uint32_t)__popc(s3);
        const uint32_t incl = wave_incl_scan_dpp(c);
        // one word per lane for the boundaries: the starts in the lanes
        // before it (< 1024, 11 bits), then those in its first one, two and
        // three dwords (<= 12 each, 5 bits)
        const uint32_t pk = (incl - c) | (c0 << 11) | (c01 << 16) | (c012 << 21);
        carry = readlane32(h3, 63) >> 31;
        uint32_t fbr = 0, pend = 0;   // forced starts before P / at the last P
        uint32_t lastP = ~0u;
        while (rem) {
            const int j = __ffsll((unsigned long long)rem) - 1;
            const uint32_t P = readlane32(wrel, j);
            if (P >= (u + 1u) * kRound) break;
            rem &= rem - 1;
            const uint32_t rel = P - u * kRound;
            const int L = (int)(rel >> 4);
            const uint32_t r = rel & 15u, k = r >> 2, sh = 8u * (r & 3u);
            // lane L's dword k: its start bits and whitespace bits
            uint32_t wk, hk;
            if (k == 0) { wk = readlane32(s0, L); hk = readlane32(h0, L); }
            else if (k == 1) { wk = readlane32(s1, L); hk = readlane32(h1, L); }
            else if (k == 2) { wk = readlane32(s2, L); hk = readlane32(h2, L); }
            else { wk = readlane32(s3, L); hk = readlane32(h3, L); }
            if (P != lastP) {
                fbr += pend;
                lastP = P;
                // whitespace at P-1: in the same dword unless P starts it
                uint32_t prev;
                if (sh) prev = hk >> (sh - 1u);
                else if (k == 0) prev = readlane32(v0, L) >> 7;
                else if (k == 1) prev = readlane32(v1, L) >> 7;
                else if (k == 2) prev = readlane32(v2, L) >> 7;
                else prev = readlane32(v3, L) >> 7;
                pend = ((hk >> (sh + 7)) | prev) & 1u ? 0u : 1u;
            }
            const uint32_t q = readlane32(pk, L);
            const uint32_t below = k ? (q >> (6u + 5u * k)) & 31u : 0u;   // starts in dwords 0 .. k-1
            const uint32_t part = below + (uint32_t)__popc(wk & ((1u << sh) - 1u));
            const uint32_t val = (uint32_t)(base + fbr + (q & 0x7FFu) + part);
            plv = lane == j ? val : plv;
        }
        base += readlane32(incl, 63) + fbr + pend;
    }
    if ((bm >> lane) & 1ull) rc.ploc[st.wb + (uint32_t)lane] = plv;
    st.running = base;
    st.ws_prev = carry;
    st.s_ptr += (uint32_t)__popcll(bm);
}

__global__ __launch_bounds__(kBlock, 7) void k_char_main(const uint8_t *__restrict__ text, uint64_t B,
                                                      const uint64_t *__restrict__ off, uint32_t N,
                                                      uint64_t Rw, uint32_t nwaves,
                                                      uint32_t *__restrict__ ploc,
                                                      uint64_t *__restrict__ wavetot)
{
    __shared__ WaveLds lds_all[kBlock / 64];
    const int lane = lane_id();
    // the wave index, known to the compiler to be uniform across the wave
    const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane((int)(blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)));
    if (w >= nwaves) return;
    WaveLds &lds = lds_all[threadIdx.x >> 6];
    if (lane < 32) *reinterpret_cast<uint4 *>(&lds.cov[4 * lane]) = make_uint4(0u, 0u, 0u, 0u);
    RangeCtx rc;
    rc.off = off;
    rc.N = N;
    rc.ws_start = (uint64_t)w * Rw;
    rc.ws_end = rc.ws_start + Rw < B ? rc.ws_start + Rw : B;
    rc.ploc = ploc;
    if (rc.ws_start >= B) {
        if (lane == 0) wavetot[w] = 0;
        return;
    }
    WaveState st;
    const bool has_pre = rc.ws_start > 0;   // then ws_start >= Rw >= 4 KiB
    st.s_ptr = lower_bound_wave(off, (uint64_t)N + 1, has_pre ? rc.ws_start - 16 : 0, lane);
    st.wb = st.s_ptr;
    st.win = win_load(off, N, st.wb, lane);
    st.running = 0;
    st.acc = 0;
    st.ws_prev = 1;
    st.spill = 0;

    const uint64_t load_end = rc.ws_end + 16;
    const uint64_t sr_bytes = (uint64_t)kRound * kLoadRounds;
    if (has_pre) {
        // the 16 bytes before the range, in lane 63 of a round of its own:
        // they carry the whitespace state of the byte before the range and
        // any separator spilling into its first bytes (nothing is counted)
        uint64_t rb = rc.ws_start - kRound;
        uint4 dp = lane == 63 ? load16(text, B, rc.ws_start - 16) : make_uint4(0u, 0u, 0u, 0u);
        uint32_t dn_top = load4(text, B, rc.ws_start);
        process_round(st, rc, dp, dn_top, rb, lane);
    }
    for (uint64_t sb = rc.ws_start; sb < rc.ws_end; sb += sr_bytes) {
        // whole: every chunk and the trailing dword lie inside the buffer
        const bool whole = sb + sr_bytes + 4 <= B;
        uint4 d[kLoadRounds];
        uint32_t tail = 0;
        if (whole) {
#pragma unroll
            for (uint32_t u = 0; u < kLoadRounds; u++) {
                v4u v = __builtin_nontemporal_load(
                    reinterpret_cast<const v4u *>(text + sb + (uint64_t)u * kRound + 16u * (uint32_t)lane));
                d[u] = make_uint4(v.x, v.y, v.z, v.w);
            }
            tail = *reinterpret_cast<const uint32_t *>(text + sb + sr_bytes);
        } else {
#pragma unroll
            for (uint32_t u = 0; u < kLoadRounds; u++) {
                uint64_t c = sb + (uint64_t)u * kRound + 16u * (uint32_t)lane;
                d[u] = (c < load_end && c < B) ? load16(text, B, c) : make_uint4(0u, 0u, 0u, 0u);
            }
            if (sb + sr_bytes < load_end) tail = load4(text, B, sb + sr_bytes);
        }
        // Super-round paths (all bytes counted, no separator carried in):
        // with no prompt boundary before sb + 4098, multi-byte separators
        // are checked cooperatively; with boundaries but no UTF-8 lead
        // byte, they are attributed per boundary. Otherwise: per round.
        bool fast = false;
        uint64_t bm = 0;   // window lanes holding this super-round's boundaries
        if (whole && sb + sr_bytes <= rc.ws_end && st.spill == 0) {
            ensure_window(st, rc, st.s_ptr, lane);
            uint32_t kk = st.s_ptr - st.wb;
            uint64_t near = __ballot((uint32_t)lane >= kk && st.win < sb + sr_bytes + 2);
            if ((near >> 63) & 1ull) {
                // the window may end inside the super-round: restart it here
                st.wb = st.s_ptr;
                st.win = win_load(rc.off, rc.N, st.wb, lane);
                kk = 0;
                near = __ballot(st.win < sb + sr_bytes + 2);
            }
            if (!((near >> 63) & 1ull)) {
                fast = near == 0;
                bm = __ballot((uint32_t)lane >= kk && st.win < sb + sr_bytes);
            }
        }
        // lead bytes (>= 0xC0) of the super-round, listed only when some
        // byte has bit 7 set
        uint64_t M = 0;
        bool leads = false;
        if ((fast || bm) && __ballot(high_any(d) != 0)) {
            M = (uint64_t)(lead_bits(d[0]) | (lead_bits(d[1]) << 4)) |
                ((uint64_t)(lead_bits(d[2]) | (lead_bits(d[3]) << 4)) << 32);
            leads = __ballot(M != 0) != 0;
        }
        if (bm && !leads) {
            boundary_superround(st, rc, d, sb, bm, lane);
            continue;
        }
        if (fast) {
            uint32_t cov[kLoadRounds] = {0u, 0u, 0u, 0u};
            uint32_t spill_next = 0;
            int res = 1;
            if (leads) {
                const uint32_t nl = (uint32_t)__popcll(M);
                const uint32_t incl = wave_incl_scan_dpp(nl);
                res = superround_separators(lds, d, tail, M, incl - nl, readlane32(incl, 63), lane,
                                            cov, spill_next);
            }
            if (res != 0) {
                uint32_t carry = st.ws_prev;
                uint32_t acc = 0;
#pragma unroll
                for (uint32_t u = 0; u < kLoadRounds; u++) {
                    uint32_t h0 = ascii_space_hb(d[u].x), h1 = ascii_space_hb(d[u].y);
                    uint32_t h2 = ascii_space_hb(d[u].z), h3 = ascii_space_hb(d[u].w);
                    if (res == 2) {
                        h0 |= expand4(cov[u] & 0xFu);
                        h1 |= expand4((cov[u] >> 4) & 0xFu);
                        h2 |= expand4((cov[u] >> 8) & 0xFu);
                        h3 |= expand4((cov[u] >> 12) & 0xFu);
                    }
                    // lane i receives lane i-1's last dword; lane 0 the carried bit
                    uint32_t p0 = wave_shr1(h3, carry << 31);
                    uint32_t s0 = ~h0 & __builtin_amdgcn_alignbyte(h0, p0, 3);
                    uint32_t s1 = ~h1 & __builtin_amdgcn_alignbyte(h1, h0, 3);
                    uint32_t s2 = ~h2 & __builtin_amdgcn_alignbyte(h2, h1, 3);
                    uint32_t s3 = ~h3 & __builtin_amdgcn_alignbyte(h3, h2, 3);
                    acc += __popc(s0) + __popc(s1) + __popc(s2) + __popc(s3);
                    carry = readlane32(h3, 63) >> 31;
                }
                st.acc += acc;
                st.ws_prev = carry;
                st.spill = spill_next;
                continue;
            }
        }
#pragma unroll
        for (uint32_t u = 0; u < kLoadRounds; u++) {
            uint64_t rb = sb + (uint64_t)u * kRound;
            if (rb >= rc.ws_end) break;
            uint32_t dn_top = u + 1 < kLoadRounds ? readlane32(d[u + 1 < kLoadRounds ? u + 1 : u].x, 0)
                                                  : tail;
            process_round(st, rc, d[u], dn_top, rb, lane);
        }
    }
    uint64_t total = st.running + readlane32(wave_incl_scan_dpp(st.acc), 63);
    if (lane == 0) wavetot[w] = total;
}

// counts[i] from the per-boundary local prefixes and the per-wave totals:
// the word starts of [a, b) are the starts after a in a's wave, those of the
// whole waves in between, and the starts before b in b's wave.
// Per prompt: the word count from the waves' totals and the boundary
// positions; with sc.n != 0 the request is also scored (stage 3) from that
// count.
__global__ __launch_bounds__(256) void k_char_fin(const uint64_t *__restrict__ off, uint32_t N,
                                                  uint64_t B, uint32_t rw_kib, uint32_t nwaves,
                                                  const uint64_t *__restrict__ wavetot,
                                                  const uint32_t *__restrict__ ploc,
                                                  uint32_t *__restrict__ counts, ScoreArgs sc)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N;
         i += (uint64_t)gridDim.x * blockDim.x) {
        uint64_t a = off[i], b = off[i + 1];
        if (b <= a || a >= B) {
            counts[i] = 0;
            if (sc.n) score_one(sc, (uint32_t)i, 0u);
            continue;
        }
        uint32_t wa = (uint32_t)(a >> 10) / rw_kib;
        uint32_t wb;
        uint64_t tail;
        if (b >= B) {
            wb = nwaves;
            tail = 0;
        } else {
            wb = (uint32_t)(b >> 10) / rw_kib;
            tail = ploc[i + 1];
        }
        uint64_t sum = tail;
        for (uint32_t w = wa; w < wb && w < nwaves; w++) sum += wavetot[w];
        const uint32_t cnt = (uint32_t)(sum - ploc[i]);
        counts[i] = cnt;
        if (sc.n) score_one(sc, (uint32_t)i, cnt);
    }
}

// DS_VALIDATE: offsets nondecreasing and offsets[N] <= B.
__global__ void k_char_validate(const uint64_t *__restrict__ off, uint32_t N, uint64_t B,
                                uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N;
         i += (uint64_t)gridDim.x * blockDim.x)
        if (off[i] > off[i + 1]) bad = 1;
    if (blockIdx.x == 0 && threadIdx.x == 0 && off[N] > B) bad = 1;
    if (bad) atomicOr(flag, 1u);
}

// The read side of k_char_main alone: the same wave ranges and 16-byte
// nontemporal loads, four rounds in flight per wave, and no classification;
// each wave's XOR of its words goes to sink[w], so that no load is dropped.
// B is a multiple of 16.
__global__ __launch_bounds__(kBlock) void k_read_stream(const uint8_t *__restrict__ p, uint64_t B, uint64_t Rw,
                                                      uint32_t nwaves, uint32_t *__restrict__ sink)
{
    const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane((int)(blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)));
    if (w >= nwaves) return;
    const int lane = lane_id();
    const uint64_t b = (uint64_t)w * Rw, e = b + Rw < B ? b + Rw : B;
    uint32_t acc = 0;
    for (uint64_t sb = b; sb < e; sb += (uint64_t)kRound * kLoadRounds) {
        v4u d[kLoadRounds];
#pragma unroll
        for (uint32_t u = 0; u < kLoadRounds; u++) {
            const uint64_t c = sb + (uint64_t)u * kRound + 16u * (uint32_t)lane;   // c < e: c + 16 <= e
            d[u] = c < e ? __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p + c)) : v4u{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (uint32_t u = 0; u < kLoadRounds; u++) acc ^= d[u].x ^ d[u].y ^ d[u].z ^ d[u].w;
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, m, 64);
    if (lane == 0) sink[w] = acc;
}

// Wave ranges of k_char_main for B bytes: one per resident wave slot (CUs x
// resident waves of k_char_main per CU) times kRangesPerSlot, whole 4 KiB
// super-rounds.
hipError_t char_waves(uint64_t B, uint64_t &Rw, uint32_t &nwaves)
{
    static int resident_cache[64];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    int resident = dev >= 0 && dev < 64 ? resident_cache[dev] : 0;
    if (resident == 0) {
        int n_cu = 0, per_cu = 0;
        e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_char_main, kBlock, 0);
        if (e != hipSuccess) return e;
        resident = (n_cu > 0 ? n_cu : 1) * (per_cu > 0 ? per_cu : 1) * (int)(kBlock / 64);
        if (dev >= 0 && dev < 64) resident_cache[dev] = resident;
    }
    uint64_t target = (uint64_t)resident * kRangesPerSlot;
    if (target > kMaxWaves) target = kMaxWaves;
    Rw = align_up(cdiv(B ? B : 1, target), (uint64_t)kRound * kLoadRounds);
    nwaves = (uint32_t)cdiv(B, Rw);
    return hipSuccess;
}

}  // namespace

size_t char_ws_bytes(uint64_t n)
{
    return align_up((n + 1) * 4, 256) + align_up((uint64_t)kMaxWaves * 8, 256);
}

hipError_t char_launch(const uint8_t *text, uint64_t B, const uint64_t *offsets, uint32_t n,
                       uint32_t *counts, void *ws, uint32_t *flag, hipStream_t s, const ScoreArgs *score)
{
    uint8_t *p = static_cast<uint8_t *>(ws);
    uint32_t *ploc = reinterpret_cast<uint32_t *>(p);
    p += align_up(((uint64_t)n + 1) * 4, 256);
    uint64_t *wavetot = reinterpret_cast<uint64_t *>(p);

    if (flag) {
        uint32_t blocks = (uint32_t)(cdiv(n, 256) < 1024 ? cdiv(n, 256) : 1024);
        if (blocks == 0) blocks = 1;
        hipLaunchKernelGGL(k_char_validate, dim3(blocks), dim3(256), 0, s, offsets, n, B, flag);
        return hipGetLastError();
    }
    uint64_t Rw = 0;
    uint32_t nwaves = 0;
    hipError_t e = char_waves(B, Rw, nwaves);
    if (e != hipSuccess) return e;
    if (nwaves > 0) {
        uint32_t blocks = (uint32_t)cdiv(nwaves, kBlock / 64);
        hipLaunchKernelGGL(k_char_main, dim3(blocks), dim3(kBlock), 0, s, text, B, offsets, n, Rw,
                           nwaves, ploc, wavetot);
    }
    uint64_t fb = cdiv(n, 256);
    uint32_t fblocks = (uint32_t)(fb < 4096 ? fb : 4096);
    if (fblocks)
        hipLaunchKernelGGL(k_char_fin, dim3(fblocks), dim3(256), 0, s, offsets, n, B,
                           (uint32_t)(Rw >> 10), nwaves, wavetot, ploc, counts,
                           score ? *score : ScoreArgs{});
    return hipGetLastError();
}

hipError_t readbw_launch(const void *buf, uint64_t bytes, uint32_t *xor_out, hipStream_t s)
{
    hipError_t e = fill_u32(xor_out, 0u, kReadBwWords, s);   // a fill kernel, not a memset
    if (e != hipSuccess || bytes == 0) return e;
    uint64_t Rw = 0;
    uint32_t nwaves = 0;
    e = char_waves(bytes, Rw, nwaves);
    if (e != hipSuccess) return e;
    static_assert(kMaxWaves <= kReadBwWords, "a word per wave");
    const uint32_t blocks = (uint32_t)cdiv(nwaves, kBlock / 64);
    hipLaunchKernelGGL(k_read_stream, dim3(blocks), dim3(kBlock), 0, s, static_cast<const uint8_t *>(buf), bytes, Rw,
                       nwaves, xor_out);
    return hipGetLastError();
}

}  // namespace ds
