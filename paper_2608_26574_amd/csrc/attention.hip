// State-masked attention over the augmented block (Sec. 3.1, Sec. 3.2).
//
// bf16 path: flash-style on v_mfma_f32_32x32x16_bf16.  A workgroup serves
// 32 * WAVES query rows that read one KV head -- with grouped-query attention
// the rows of all query heads of that KV head are one row space, so a K/V
// tile staged once in LDS feeds every head of the group -- with G groups of
// WAVES waves that take interleaved 64-key tiles (merged through LDS at the
// end).  The V cache is stored dims-major (V^T, [dh][cap] per KV head), so
// both tiles of a step are plain copies: every lane moves 16-byte chunks from
// global memory straight into LDS (global_load_lds).  Chunks are XOR-swizzled
// by row so the MFMA operand reads are bank-conflict free.  With two key
// groups, the second runs half a tile step out of phase (its softmax while
// the first group's scores run on the matrix cores, and the reverse), so the
// two waves sharing a SIMD overlap MFMA and VALU work.
// Each wave owns 32 query rows:
//   S^T = K * Q^T   (A = 32 keys from LDS, B = this wave's Q rows in registers)
//   O^T += V^T P^T  (A = V^T from LDS, B = probabilities straight from the
//                    S^T accumulators)
// Lane l supplies A row l%32 of S^T with key pi(l%32), pi swapping bits 2 and
// 3, so that the 8 probabilities a lane holds for each 16-key step of O^T are
// 8 consecutive keys and the matching V^T operand is one 16-byte read.
// Keys are tiled in two runs: the prefix [0, P) in 64-key tiles, then the
// block [P, P + 2B) (x^j at P+j, s^j at P+B+j) in 64-key tiles of its own.  A
// row's block visibility is the "take x" word of the state mask (Eq. 2-3,
// built once per step) widened to 2B bits: x^j where the bit is set, s^j
// where it is clear; so one aligned 64-bit word per block tile says which
// keys a row sees, and full prefix tiles need no test at all.
// The softmax runs in the log2 domain against a running maximum that may lag
// the true one: a tile's probabilities are taken against the running maximum
// as it stands, and only when a lane's sum of them exceeds kBig = 256 (always
// on a row's first visible tile, where the running maximum is still the
// floor; and whenever a score exceeds the running maximum by more than 8) is
// the tile's maximum taken, the accumulators rescaled and the probabilities
// recomputed.  A tile needs no maximum reduction otherwise.
// Long key ranges may also be split across workgroups (fp32 partials of
// (o, m, l), merged in split order by a small combine kernel).
//
// fp32 path: one thread per (row, head), plain online softmax.
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace dard {

namespace {

constexpr int kKeys = 64;      // keys per tile
constexpr int kMaxSplit = 16;  // key splits across workgroups
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kMinLog2 = -1e30f;   // running-max floor (log2 units): exp2 of anything below it is 0
constexpr float kBig = 256.f;        // a lane's probability sum over a tile that moves the running max

// LDS of one group of TPG threads: three K stages [64 keys][DH] and two V^T
// stages [DH][64 keys], unpadded and XOR-swizzled in 16-byte chunks, or, at
// the end, every lane's o, m and l for the merge of the groups.
template <int DH, int TPG>
struct Lds {
    static constexpr int TILE = kKeys * DH * 2;    // bytes of one K or V^T tile
    static constexpr int MERGE = (DH / 2 + 2) * TPG * 4;
    static constexpr int GROUP = ((5 * TILE > MERGE ? 5 * TILE : MERGE) + 15) / 16 * 16;
};

// 16-byte chunk slots.  The LDS serves a 16-byte read 16 consecutive lanes
// per cycle over 64 banks (256 bytes; measured: an image that separates only
// groups of 8 lanes within 128 bytes kept its conflicts), and each group must
// hit 16 different 4-bank groups; the swizzles below also keep every 8 lanes
// within 128 bytes apart.  With x ^ (x >> 3) a value x in [0, 16) and its
// neighbour x ^ 8 differ in their low three bits.
//   K row r keeps its chunk c (dims 8c..8c+7) in slot c ^ kswz(r): with
//   x = pi(r) % 16, pi swapping bits 2 and 3, kswz = x for DH = 128 (a row
//   is 256 bytes) and (x ^ (x >> 3)) % 8 for DH = 64.  The S^T operand read
//   of lane l takes key row pi(l % 32), so x is l % 16.
//   V^T row d (a dim, 128 bytes) keeps its chunk c (keys 8c..8c+7) in slot
//   c ^ vswz(d), vswz(d) = (d ^ (d >> 3)) % 8; the V^T read of lane l takes
//   row 32j + l % 32.
__device__ __forceinline__ int swap23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }
template <int DH>
__device__ __forceinline__ int kswz(int r) {
    const int x = swap23(r) & 15;   // rows 32 apart share their swizzle
    return DH == 128 ? x : ((x ^ (x >> 3)) & (DH / 8 - 1));
}
template <int DH>
__device__ __forceinline__ int kslot(int r, int c) { return r * (DH / 8) + (c ^ kswz<DH>(r)); }
__device__ __forceinline__ int vswz(int d) { return (d ^ (d >> 3)) & 7; }
__device__ __forceinline__ int vslot(int d, int c) { return d * (kKeys / 8) + (c ^ vswz(d)); }

// The 2B-bit block visibility of a row, x^j for the set bits j of its take-x
// value X (B <= 256 bits, zero above B), s^j for the clear ones: bits [0, B)
// are X, bits [B, 2B) are NOT X.  block_word gives bits [64 bt, 64 bt + 64),
// the word of block tile bt.
__device__ __forceinline__ uint64_t word_at(const uint64_t (&x)[kBlockWords], int q) {
    uint64_t w = 0ull;
#pragma unroll
    for (int k = 0; k < kBlockWords; ++k) w = q == k ? x[k] : w;
    return w;
}
// Bits [start, start + 64) of X (start may be negative), zero outside [0, B).
__device__ __forceinline__ uint64_t bits64(const uint64_t (&x)[kBlockWords], int B, int start) {
    if (start >= B || start <= -64) return 0ull;
    uint64_t v;
    if (start < 0) {
        v = word_at(x, 0) << (-start);
    } else {
        const int q = start >> 6, sh = start & 63;
        v = word_at(x, q) >> sh;
        if (sh) v |= word_at(x, q + 1) << (64 - sh);
    }
    const int n = B - start;
    return n < 64 ? v & ((1ull << n) - 1) : v;
}
// Bits j of a word with 0 <= start + j < B.
__device__ __forceinline__ uint64_t range_mask(int start, int B) {
    const int lo = start < 0 ? -start : 0;
    const int hi = B - start < 64 ? B - start : 64;
    if (hi <= lo) return 0ull;
    const uint64_t up = hi >= 64 ? ~0ull : (1ull << hi) - 1;
    const uint64_t low = lo >= 64 ? ~0ull : (1ull << lo) - 1;
    return up & ~low;
}
__device__ __forceinline__ uint64_t block_word(const uint64_t (&x)[kBlockWords], int B, int bt) {
    const int s0 = 64 * bt;
    return bits64(x, B, s0) | (~bits64(x, B, s0 - B) & range_mask(s0 - B, B));
}

// First key and key count of tile t (npre prefix tiles over [0, pre_end),
// then block tiles over [P, P + 2B)).
__device__ __forceinline__ int tile_first(int t, int npre, int P) { return t < npre ? t * kKeys : P + (t - npre) * kKeys; }
__device__ __forceinline__ int tile_count(int t, int npre, int pre_end, int B2) {
    return t < npre ? min(kKeys, pre_end - t * kKeys) : min(kKeys, B2 - (t - npre) * kKeys);
}

// Grid: x = row tile (row tile fastest, then KV head, then sequence), dealt to
// the XCDs in contiguous runs so the workgroups reading one KV head share an
// L2; y = key split.
// KV8: the cache holds OCP FP8 E4M3 codes; tiles go through registers (8
// bytes per 8-key or 8-dim chunk), are widened to bf16 and written to LDS in
// the same swizzled image the bf16 copies produce, so the MFMA code is shared.
template <int DH, int WAVES, int G, bool KV8>
__global__ __launch_bounds__(64 * WAVES * G) __attribute__((amdgpu_waves_per_eu(G)))
void attn_mfma_kernel(AttnArgs a, int rowtiles, int tps) {
    constexpr int TPG = 64 * WAVES, ROWS = 32 * WAVES;
    constexpr int NCH = kKeys * DH / 8;            // 16-byte chunks per K (and per V^T) tile
    constexpr int NI = NCH / TPG;                  // chunks per thread per tile, each
    static_assert(NCH % TPG == 0, "whole chunks per thread");
    using L = Lds<DH, TPG>;
    typedef __attribute__((address_space(3))) void* lds_ptr;
    typedef __attribute__((address_space(1))) void* glb_ptr;
    __shared__ __attribute__((aligned(16))) char smem[G * L::GROUP];

    // group and wave are wave-uniform: say so, so that tile bookkeeping stays scalar
    const int grp = __builtin_amdgcn_readfirstlane(threadIdx.x / TPG), tid = threadIdx.x % TPG;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 31, eta = lane >> 5;
    int bid = blockIdx.x;
    const int total = gridDim.x;
    if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
    const int split = blockIdx.y, nsplit = gridDim.y;
    const int rt = bid % rowtiles;
    const int kvh = (bid / rowtiles) % a.Hkv;
    const int s = bid / rowtiles / a.Hkv;
    const int GQ = a.Hq / a.Hkv;
    const int nrows = GQ * a.R;

    // prefix tiles [0, npre), then block tiles (masked mode)
    const int pre_end = a.masked ? a.P : a.nkeys;
    const int npre = (pre_end + kKeys - 1) / kKeys;
    const int ntiles = npre + (a.masked ? (2 * a.B + kKeys - 1) / kKeys : 0);
    const int t_begin = split * tps;
    const int t_end = min(ntiles, t_begin + tps);
    const int iters = (t_end - t_begin + G - 1) / G;   // tile steps of every group
    const int P = a.P, B2 = 2 * a.B, cap = a.cap;

    using KVT = typename std::conditional<KV8, uint8_t, bf16_t>::type;
    const KVT* kbase = reinterpret_cast<const KVT*>(a.k) + ((size_t)s * a.Hkv + kvh) * cap * DH;
    const KVT* vbase = reinterpret_cast<const KVT*>(a.v) + ((size_t)s * a.Hkv + kvh) * DH * cap;
    // keys below P_sh (whole tiles) come from the cache the batch shares
    const KVT* kbase_sh = a.P_sh ? reinterpret_cast<const KVT*>(a.k_sh) + (size_t)kvh * a.cap_sh * DH : kbase;
    const KVT* vbase_sh = a.P_sh ? reinterpret_cast<const KVT*>(a.v_sh) + (size_t)kvh * DH * a.cap_sh : vbase;
    char* gbase = smem + grp * L::GROUP;

    // ---- copy the K (or V^T) tile of key tile `tile` into LDS at `dst`:
    // chunk q = (wave * NI + j) * 64 + lane of the swizzled image, straight to
    // LDS.  In a ragged tile (n < 64 keys) nothing past the valid keys is read:
    // K rows past n are skipped (their scores are masked, whatever the stage
    // held), V^T chunks past n are written as zeros (their probabilities are 0
    // and 0 * stale could be NaN), and a chunk that straddles n goes through
    // registers element by element.
    // FP8 cache: this thread's chunks of the next K and V tiles, held in
    // registers between their loads (early in a step) and their conversion
    // into LDS (at the end of the step, before its barrier)
    uint2 kreg[NI], vreg[NI];
    auto load_k8 = [&](int tile) __attribute__((always_inline)) {
        const int k0 = tile_first(tile, npre, P), n = tile_count(tile, npre, pre_end, B2);
        const KVT* kb = k0 < a.P_sh ? kbase_sh : kbase;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int q = (wave * NI + j) * 64 + lane;
            const int r = q / (DH / 8), sl = q % (DH / 8);
            // a key row of DH bytes: every 8-byte chunk is aligned
            if (n == kKeys || r < n)
                kreg[j] = *reinterpret_cast<const uint2*>(kb + (size_t)(k0 + r) * DH + 8 * (sl ^ kswz<DH>(r)));
        }
    };
    auto commit_k8 = [&](int tile, char* dst) __attribute__((always_inline)) {
        const int n = tile_count(tile, npre, pre_end, B2);
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int q = (wave * NI + j) * 64 + lane;
            if (n == kKeys || q / (DH / 8) < n) *reinterpret_cast<uint4*>(dst + 16 * q) = e4m3x8_to_bf16x8(kreg[j]);
        }
    };
    auto load_v8 = [&](int tile) __attribute__((always_inline)) {
        const int k0 = tile_first(tile, npre, P), n = tile_count(tile, npre, pre_end, B2);
        const bool sh = k0 < a.P_sh;
        const KVT* vb = sh ? vbase_sh : vbase;
        const int vcap = sh ? a.cap_sh : cap;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int q = (wave * NI + j) * 64 + lane;
            const int d = q / (kKeys / 8), c = (q % (kKeys / 8)) ^ vswz(d);
            const KVT* src = vb + (size_t)d * vcap + k0 + 8 * c;
            const int cnt = n == kKeys ? 8 : max(0, min(8, n - 8 * c));   // keys of the chunk inside the tile
            uint2 w = make_uint2(0u, 0u);                                    // code 0 is +0
            if (cnt == 8 && ((reinterpret_cast<uintptr_t>(src) & 7) == 0)) {
                w = *reinterpret_cast<const uint2*>(src);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (e < cnt) {
                        const uint32_t bt = (uint32_t)src[e] << (8 * (e & 3));
                        if (e < 4) w.x |= bt; else w.y |= bt;
                    }
            }
            vreg[j] = w;
        }
    };
    auto commit_v8 = [&](char* dst) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int q = (wave * NI + j) * 64 + lane;
            *reinterpret_cast<uint4*>(dst + 16 * q) = e4m3x8_to_bf16x8(vreg[j]);
        }
    };
    // byte offsets of this thread's chunks inside a K tile and inside a V^T
    // tile of the sequence's own cache (the same for every tile)
    uint32_t koff[NI], voff[NI];
#pragma unroll
    for (int j = 0; j < NI; ++j) {
        const int q = (wave * NI + j) * 64 + lane;
        const int r = q / (DH / 8), d = q / (kKeys / 8);
        koff[j] = (uint32_t)(r * DH + 8 * ((q % (DH / 8)) ^ kswz<DH>(r))) * sizeof(KVT);
        voff[j] = (uint32_t)(d * cap + 8 * ((q % (kKeys / 8)) ^ vswz(d))) * sizeof(KVT);
    }
    auto issue_k = [&](int tile, char* dst) __attribute__((always_inline)) {
        if constexpr (KV8) {
            load_k8(tile);
            commit_k8(tile, dst);
        } else {
        const int k0 = tile_first(tile, npre, P), n = tile_count(tile, npre, pre_end, B2);
        const KVT* kb = k0 < a.P_sh ? kbase_sh : kbase;
        if (n == kKeys) {   // a full tile: the common case, no per-chunk test
            const char* kt = reinterpret_cast<const char*>(kb + (size_t)k0 * DH);
#pragma unroll
            for (int j = 0; j < NI; ++j)
                __builtin_amdgcn_global_load_lds((glb_ptr)(kt + koff[j]), (lds_ptr)(dst + (wave * NI + j) * 1024),
                                                 16, 0, 0);
            return;
        }
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int q = (wave * NI + j) * 64 + lane;
            const int r = q / (DH / 8), sl = q % (DH / 8);
            const KVT* src = kb + (size_t)(k0 + r) * DH + 8 * (sl ^ kswz<DH>(r));
            if (r < n)
                __builtin_amdgcn_global_load_lds((glb_ptr)src, (lds_ptr)(dst + (wave * NI + j) * 1024), 16, 0, 0);
        }
        }
    };
    auto issue_v = [&](int tile, char* dst) __attribute__((always_inline)) {
        if constexpr (KV8) {
            load_v8(tile);
            commit_v8(dst);
        } else {
        const int k0 = tile_first(tile, npre, P), n = tile_count(tile, npre, pre_end, B2);
        const bool sh = k0 < a.P_sh;
        if (n == kKeys && !sh) {   // a full tile of the own cache: no per-chunk test
            const char* vt = reinterpret_cast<const char*>(vbase + k0);
#pragma unroll
            for (int j = 0; j < NI; ++j)
                __builtin_amdgcn_global_load_lds((glb_ptr)(vt + voff[j]), (lds_ptr)(dst + (wave * NI + j) * 1024),
                                                 16, 0, 0);
            return;
        }
        const KVT* vb = sh ? vbase_sh : vbase;
        const int vcap = sh ? a.cap_sh : cap;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int q = (wave * NI + j) * 64 + lane;
            const int d = q / (kKeys / 8), c = (q % (kKeys / 8)) ^ vswz(d);
            const KVT* src = vb + (size_t)d * vcap + k0 + 8 * c;
            if (n == kKeys || 8 * c + 8 <= n) {
                __builtin_amdgcn_global_load_lds((glb_ptr)src, (lds_ptr)(dst + (wave * NI + j) * 1024), 16, 0, 0);
            } else {
                bf16x8 vv = {};
                if (8 * c < n) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (8 * c + e < n) vv[e] = __builtin_bit_cast(__bf16, src[e]);
                }
                *reinterpret_cast<bf16x8*>(dst + 16 * q) = vv;
            }
        }
        }
    };
    // stage addresses by arithmetic on the LDS array (an indexed table of
    // pointers would lose the address space and turn LDS reads into flat loads)
    auto kst = [&](int i) __attribute__((always_inline)) { return gbase + (i % 3) * L::TILE; };
    auto vst = [&](int i) __attribute__((always_inline)) { return gbase + (3 + (i & 1)) * L::TILE; };
    auto tile_of = [&](int it) __attribute__((always_inline)) { return t_begin + grp + G * it; };
    // A ragged K tile's copies skip the rows past its end, so a wave may issue
    // fewer than NI of them; the end-of-step wait then counts on the newest K
    // tile's NI copies only when that tile is full, and otherwise waits for
    // every copy (an older copy must never be left in flight at the barrier).
    auto full_tile = [&](int tile) __attribute__((always_inline)) {
        return tile_count(tile, npre, pre_end, B2) == kKeys;
    };
    auto mine = [&](int it) __attribute__((always_inline)) { return it < iters && tile_of(it) < t_end; };
    if (mine(0)) {
        issue_k(tile_of(0), kst(0));
        issue_v(tile_of(0), vst(0));
    }

    // ---- this lane's query row (rows of every query head of the KV head form
    // one row space), its Q fragments (B operand chunk c = dims 16c + 8eta ..)
    // and its block visibility
    const int rho = rt * ROWS + 32 * wave + lr;
    const bool row_ok = rho < nrows;
    const int h = kvh * GQ + (row_ok ? rho / a.R : 0);
    const int r = row_ok ? rho % a.R : 0;
    bf16x8 qf[DH / 16];
    {
        const bf16_t* qp = reinterpret_cast<const bf16_t*>(a.q) + (((size_t)s * a.R + r) * a.Hq + h) * DH;
#pragma unroll
        for (int c = 0; c < DH / 16; ++c) {
            bf16x8 z = {};
            qf[c] = row_ok ? ld_bf16x8(qp + 16 * c + 8 * eta) : z;
        }
    }
    uint64_t xw[kBlockWords];     // the row's take-x words
#pragma unroll
    for (int q = 0; q < kBlockWords; ++q) xw[q] = 0ull;
    if (a.masked && row_ok) {
        const int W = (a.B + 63) / 64;
        if (r < a.ctx_rows) {   // outside the block: every x key, no shadow key
#pragma unroll
            for (int q = 0; q < kBlockWords; ++q) xw[q] = block_word_mask(a.B, q);
        } else {
            const uint64_t* sp = a.sel + ((size_t)s * (a.R - a.ctx_rows) + (r - a.ctx_rows)) * W;
#pragma unroll
            for (int q = 0; q < kBlockWords; ++q)
                if (q < W) xw[q] = sp[q];
        }
    }
    const float sl2 = a.scale * kLog2e;
    // K row this lane supplies to the S^T MFMAs: key pi(lr) of each 32-key
    // block.  Operand addresses inside a stage: K chunk 2c + eta of key block
    // kb is at kaddr0 ^ 32c, plus kb * 32 rows (kswz repeats every 32 rows);
    // V^T chunk 2st + eta of dim block d at (vaddr0 ^ 32 (st ^ 2 (d & 1))) +
    // d * 32 rows (vswz(32 + x) = vswz(x) ^ 4 for x < 32).  The XOR touches
    // bits 5-6 (5-7) only, below a row and above the eta chunk, and the stage
    // bases are multiples of 16 KB, so base + (addr0 ^ m) = (base + addr0) ^ m:
    // a step adds the stage base once per operand and XORs per chunk, and the
    // block steps are immediate offsets.
    const int krow = swap23(lr);
    const uint32_t kaddr0 = 16 * kslot<DH>(krow, eta), vaddr0 = 16 * vslot(lr, eta);

    floatx16 o[DH / 32];
#pragma unroll
    for (int d = 0; d < DH / 32; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[d][v] = 0.f;
    float m_run = kMinLog2, l_run = 0.f;

    // ---- S^T = K * Q^T for the K tile at ks: value v of block kb is key
    // 32kb + 16(v/8) + 8eta + v%8 of the tile
    // Each block's DH/16 operand reads are issued together ahead of its MFMAs
    // (left to itself the compiler waits for each read right before its MFMA).
    auto scores = [&](const char* ks, floatx16 (&sc)[2]) __attribute__((always_inline)) {
        constexpr int NC = DH / 16;
        const uint32_t kb0 = (uint32_t)(ks - smem) + kaddr0;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            bf16x8 kf[NC];
#pragma unroll
            for (int c = 0; c < NC; ++c)
                kf[c] = *reinterpret_cast<const bf16x8*>(smem + ((kb0 ^ (32u * c)) + kb * 32 * DH * 2));
#pragma unroll
            for (int v = 0; v < 16; ++v) sc[kb][v] = 0.f;
#pragma unroll
            for (int c = 0; c < NC; ++c) sc[kb] = mfma32x32x16(kf[c], qf[c], sc[kb]);
            __builtin_amdgcn_sched_group_barrier(0x100, NC, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, NC, 0);
        }
    };
    // ---- mask, online softmax and O^T += V^T P^T for tile `tile`
    auto softmax_pv = [&](floatx16 (&sc)[2], int tile, const char* vs) __attribute__((always_inline)) {
        // visibility: only tiles with block keys or a ragged end test it
        // (tile and n are wave-uniform, so this is a scalar branch)
        const int n = tile_count(tile, npre, pre_end, B2);
        if (!(tile < npre && n == kKeys)) {
            uint64_t vis;
            if (tile < npre) {
                vis = (1ull << n) - 1;     // n < 64 here
            } else {
                vis = block_word(xw, a.B, tile - npre);
            }
            const uint64_t ww = vis >> (8 * eta);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (!((ww >> (32 * kb + 16 * (v >> 3) + (v & 7))) & 1ull)) sc[kb][v] = -INFINITY;
        }
        // online softmax in the log2 domain, against the running maximum as
        // it stands; a tile with a row whose probabilities grow large (sum over
        // the lane's keys above kBig, also the first visible tile, where the
        // running maximum is still the floor) is recomputed after moving the
        // running maximum to the tile's maximum
        float psum = 0.f;
        bf16x8 pb[2][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float p = __builtin_amdgcn_exp2f(fmaf(sc[kb][v], sl2, -m_run));
                psum += p;
                pb[kb][v >> 3][v & 7] = (__bf16)p;
            }
        if (__ballot(psum > kBig)) {
            float mt = sc[0][0];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[kb][v]);
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float m_new = fmaxf(m_run, mt * sl2);     // sl2 > 0: the max commutes with the scale
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
            for (int d = 0; d < DH / 32; ++d) o[d] *= alpha;
            l_run *= alpha;
            m_run = m_new;
            psum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float p = __builtin_amdgcn_exp2f(fmaf(sc[kb][v], sl2, -m_run));
                    psum += p;
                    pb[kb][v >> 3][v & 7] = (__bf16)p;
                }
        }
        l_run += psum;
        // O^T += V^T * P^T: step st = 2kb + hh covers keys 16st + [0, 16); the
        // lane's 8 probabilities are keys 16st + 8eta + [0, 8), V^T chunk 2st + eta
        const uint32_t vb0 = (uint32_t)(vs - smem) + vaddr0;
#pragma unroll
        for (int d = 0; d < DH / 32; ++d) {
            bf16x8 vf[4];
#pragma unroll
            for (int st = 0; st < 4; ++st)
                vf[st] = *reinterpret_cast<const bf16x8*>(
                    smem + ((vb0 ^ (32u * (st ^ (2 * (d & 1))))) + d * 32 * kKeys * 2));
#pragma unroll
            for (int st = 0; st < 4; ++st) o[d] = mfma32x32x16(vf[st], pb[st >> 1][st & 1], o[d]);
            __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        }
    };

    // ---- main loop.  Group 0 computes step it as scores, softmax, P V; a
    // second group runs half a step out of phase -- softmax and P V of step it,
    // then the scores of step it + 1 -- so that on every SIMD one wave's MFMAs
    // overlap the other's softmax.  Copies run ahead of use: V one step, K two
    // steps (three for the second group, whose scores come a step early), so a
    // copy's latency spans more than one step.  Each step ends by waiting for
    // every copy except the newest K tile and publishing them with the barrier,
    // which also retires every wave's reads of the stages the next step
    // overwrites.  Copies complete in issue order, so V goes first.
    const bool late = G > 1 && grp == 1;
    if (mine(1)) issue_k(tile_of(1), kst(1));
    if (late && mine(2)) issue_k(tile_of(2), kst(2));
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (!late) {
        for (int it = 0; it < iters; ++it) {         // iters is uniform across the workgroup
            const bool nextv = mine(it + 1), ahead = mine(it + 2);
            if constexpr (KV8) {
                if (nextv) load_v8(tile_of(it + 1));
                if (ahead) load_k8(tile_of(it + 2));
            } else {
                if (nextv) issue_v(tile_of(it + 1), vst(it + 1));
                if (ahead) issue_k(tile_of(it + 2), kst(it + 2));
            }
            if (mine(it)) {
                floatx16 sc[2];
                scores(kst(it), sc);
                softmax_pv(sc, tile_of(it), vst(it));
            }
            if constexpr (KV8) {
                if (nextv) commit_v8(vst(it + 1));
                if (ahead) commit_k8(tile_of(it + 2), kst(it + 2));
                __builtin_amdgcn_s_waitcnt(0);
            } else {
                if (ahead && full_tile(tile_of(it + 2))) __builtin_amdgcn_s_waitcnt(waitcnt_vm(NI));
                else __builtin_amdgcn_s_waitcnt(0);
            }
            wg_barrier();
        }
    } else {
        floatx16 sc[2];
        if (mine(0)) scores(kst(0), sc);
        for (int it = 0; it < iters; ++it) {
            const bool nextv = mine(it + 1), ahead = mine(it + 3);
            if constexpr (KV8) {
                if (nextv) load_v8(tile_of(it + 1));
                if (ahead) load_k8(tile_of(it + 3));
            } else {
                if (nextv) issue_v(tile_of(it + 1), vst(it + 1));
                if (ahead) issue_k(tile_of(it + 3), kst(it + 3));
            }
            if (mine(it)) softmax_pv(sc, tile_of(it), vst(it));
            __builtin_amdgcn_sched_barrier(0);
            if (mine(it + 1)) scores(kst(it + 1), sc);
            if constexpr (KV8) {
                if (nextv) commit_v8(vst(it + 1));
                if (ahead) commit_k8(tile_of(it + 3), kst(it + 3));
                __builtin_amdgcn_s_waitcnt(0);
            } else {
                if (ahead && full_tile(tile_of(it + 3))) __builtin_amdgcn_s_waitcnt(waitcnt_vm(NI));
                else __builtin_amdgcn_s_waitcnt(0);
            }
            wg_barrier();
        }
    }

    // ---- merge the groups through LDS (group 0 keeps the result)
    if constexpr (G > 1) {
        float* mb = reinterpret_cast<float*>(gbase);
        if (grp > 0) {
#pragma unroll
            for (int d = 0; d < DH / 32; ++d)
#pragma unroll
                for (int v = 0; v < 16; ++v) mb[(16 * d + v) * TPG + tid] = o[d][v];
            mb[(DH / 2) * TPG + tid] = m_run;
            mb[(DH / 2 + 1) * TPG + tid] = l_run;
        }
        __syncthreads();
        if (grp == 0) {
            float M = m_run;
#pragma unroll
            for (int gg = 1; gg < G; ++gg)
                M = fmaxf(M, reinterpret_cast<const float*>(smem + gg * L::GROUP)[(DH / 2) * TPG + tid]);
            const float f0 = __builtin_amdgcn_exp2f(m_run - M);
            float lsum = l_run * f0;
#pragma unroll
            for (int d = 0; d < DH / 32; ++d) o[d] *= f0;
#pragma unroll
            for (int gg = 1; gg < G; ++gg) {
                const float* ob = reinterpret_cast<const float*>(smem + gg * L::GROUP);
                const float f = __builtin_amdgcn_exp2f(ob[(DH / 2) * TPG + tid] - M);
                lsum += ob[(DH / 2 + 1) * TPG + tid] * f;
#pragma unroll
                for (int d = 0; d < DH / 32; ++d)
#pragma unroll
                    for (int v = 0; v < 16; ++v) o[d][v] += ob[(16 * d + v) * TPG + tid] * f;
            }
            m_run = M;
            l_run = lsum;
        }
    }
    if (grp != 0) return;

    // ---- epilogue: the two lanes of a row hold disjoint keys; sum their l.
    // The lane holds dims 32d + 8j + 4eta + {0..3} (O^T accumulator rows).
    const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    if (!row_ok) return;
    const size_t orow = ((size_t)s * a.R + r) * a.Hq + h;    // (sequence, row, head)
    if (nsplit == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        const int tok = s * a.R + r, KO = a.Hq * DH;
        bf16_t* out = reinterpret_cast<bf16_t*>(a.out);
#pragma unroll
        for (int d = 0; d < DH / 32; ++d)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t w0 = (uint32_t)f2bf(o[d][4 * j] * inv) | ((uint32_t)f2bf(o[d][4 * j + 1] * inv) << 16);
                const uint32_t w1 = (uint32_t)f2bf(o[d][4 * j + 2] * inv) | ((uint32_t)f2bf(o[d][4 * j + 3] * inv) << 16);
                const int k = 32 * d + 8 * j + 4 * eta;
                *reinterpret_cast<uint2*>(out + (a.out_frag ? frag_off(tok, h * DH + k, KO) : orow * DH + k)) =
                    make_uint2(w0, w1);
            }
        return;
    }
    const size_t nrow = (size_t)a.b * a.R * a.Hq;
    float* po = a.part + ((size_t)split * nrow + orow) * DH;
#pragma unroll
    for (int d = 0; d < DH / 32; ++d)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            *reinterpret_cast<float4*>(po + 32 * d + 8 * j + 4 * eta) =
                make_float4(o[d][4 * j], o[d][4 * j + 1], o[d][4 * j + 2], o[d][4 * j + 3]);
    if (eta == 0) *reinterpret_cast<float2*>(a.part_ml + ((size_t)split * nrow + orow) * 2) = make_float2(m_run, l_tot);
}

// Merge key splits: O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), in split
// order.  One thread per (row, head, 4 dims); every load is issued up front.
template <int DH>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part,
                                                           const float* __restrict__ part_ml, int ns,
                                                           size_t nrow, int Hq, int frag,
                                                           bf16_t* __restrict__ out) {
    const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t row = t / (DH / 4);
    const int q4 = t % (DH / 4);
    if (row >= nrow) return;
    float m[kMaxSplit], l[kMaxSplit];
    float4 ov[kMaxSplit];
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) {
        if (sp < ns) {
            const float2 ml = reinterpret_cast<const float2*>(part_ml)[sp * nrow + row];
            m[sp] = ml.x;
            l[sp] = ml.y;
            ov[sp] = reinterpret_cast<const float4*>(part + (sp * nrow + row) * DH)[q4];
        } else {
            m[sp] = kMinLog2;
            l[sp] = 0.f;
            ov[sp] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    float M = kMinLog2;
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) M = fmaxf(M, m[sp]);
    float Lsum = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) {
        const float f = __builtin_amdgcn_exp2f(m[sp] - M);
        Lsum += l[sp] * f;
        acc.x += ov[sp].x * f; acc.y += ov[sp].y * f; acc.z += ov[sp].z * f; acc.w += ov[sp].w * f;
    }
    const float inv = Lsum > 0.f ? 1.f / Lsum : 0.f;
    const uint32_t w0 = (uint32_t)f2bf(acc.x * inv) | ((uint32_t)f2bf(acc.y * inv) << 16);
    const uint32_t w1 = (uint32_t)f2bf(acc.z * inv) | ((uint32_t)f2bf(acc.w * inv) << 16);
    const size_t o = frag ? frag_off((int)(row / Hq), (int)(row % Hq) * DH + 4 * q4, Hq * DH) : row * DH + 4 * q4;
    *reinterpret_cast<uint2*>(out + o) = make_uint2(w0, w1);
}

// fp32 path: one thread per (sequence, row, head).
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)a.b * a.R * a.Hq;
    if (t >= total) return;
    const int h = t % a.Hq;
    const int r = (t / a.Hq) % a.R;
    const int s = t / ((size_t)a.Hq * a.R);
    const int kvh = h / (a.Hq / a.Hkv);
    const float* q = reinterpret_cast<const float*>(a.q) + t * DH;
    const float* kb = reinterpret_cast<const float*>(a.k) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;
    const float* vb = reinterpret_cast<const float*>(a.v) + ((size_t)s * a.Hkv + kvh) * a.cap * DH;
    const float* kb_sh = a.P_sh ? reinterpret_cast<const float*>(a.k_sh) + (size_t)kvh * a.cap_sh * DH : kb;
    const float* vb_sh = a.P_sh ? reinterpret_cast<const float*>(a.v_sh) + (size_t)kvh * a.cap_sh * DH : vb;
    float qr[DH], o[DH];
    for (int e = 0; e < DH; ++e) { qr[e] = q[e]; o[e] = 0.f; }
    float m = -INFINITY, l = 0.f;
    // rows before ctx_rows lie outside the block: x keys only
    const bool ctx = a.masked && r < a.ctx_rows;
    const int rb = r - a.ctx_rows;
    const int i = a.masked && !ctx ? rb % a.B : 0;
    const bool shadow = a.masked && !ctx && rb >= a.B;
    const uint8_t* st = a.masked ? a.state + (size_t)s * a.B : nullptr;
    const float* cf = a.masked ? a.conf + (size_t)s * a.B : nullptr;
    for (int key = 0; key < a.nkeys; ++key) {
        if (a.masked && key >= a.P) {
            const int j = key - a.P;
            const int jj = j < a.B ? j : j - a.B;
            const bool bx = ctx || take_x(st[i], st[jj], cf[i], cf[jj], i, jj, shadow, a.flags);
            if (bx != (j < a.B)) continue;
        }
        const bool sh = key < a.P_sh;
        const float* kk = sh ? kb_sh : kb;
        const float* vv = sh ? vb_sh : vb;
        const int vcap = sh ? a.cap_sh : a.cap;
        float sdot = 0.f;
        for (int e = 0; e < DH; ++e) sdot += qr[e] * kk[(size_t)key * DH + e];
        sdot *= a.scale;
        const float mn = fmaxf(m, sdot);
        const float alpha = expf(m - mn);
        const float p = expf(sdot - mn);
        l = l * alpha + p;
        for (int e = 0; e < DH; ++e) o[e] = o[e] * alpha + p * vv[(size_t)e * vcap + key];
        m = mn;
    }
    float* out = reinterpret_cast<float*>(a.out) + t * DH;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    for (int e = 0; e < DH; ++e) out[e] = o[e] * inv;
}

// Shape of a bf16 launch (kernel-trace sweeps at the workload shapes):
// - more than 64 rows per KV head (grouped-query attention, prefill): 4 waves
//   per group, and a second, phase-shifted key group while the workgroups
//   alone leave SIMDs idle (7B GQA shape, batch 8: 35.6 -> 31.4 us);
// - 64 rows (one MHA head's augmented block): with at least 256 workgroups,
//   2 waves per workgroup (batch 16: 36 us); with few heads (batch 1-2), 4
//   waves and key splits of about 3 tiles merged by the combine kernel
//   (batch 1, prompt 736: 34 -> 20 us); in between (batch 4), no split and a
//   second key group of 2 waves taking alternate tiles (43 -> 35 us).
struct AttnCfg {
    int waves, g, rowtiles, ns, tps;
};

AttnCfg attention_cfg(int b, int R, int Hq, int Hkv, int ntiles) {
    AttnCfg c{};
    const int nrows = (Hq / Hkv) * R;
    c.g = 1;
    c.ns = 1;
    if (nrows > 64) {
        c.waves = 4;
        c.rowtiles = (nrows + 127) / 128;
        const long wgs = (long)b * Hkv * c.rowtiles;
        if (wgs * 4 < 1024 && ntiles >= 4) c.g = 2;
    } else {
        c.rowtiles = 1;
        c.waves = 2;
        const long wgs = (long)b * Hkv;
        const long by_tiles = (ntiles + 2) / 3;
        if (wgs < 256 && wgs * by_tiles <= 256) {
            // few heads: key splits of about three tiles merged by the combine
            // kernel, 4 waves per workgroup (the extra two only copy tiles)
            c.waves = 4;
            c.ns = (int)(by_tiles < kMaxSplit ? by_tiles : kMaxSplit);
        } else if (wgs < 256) {
            // more heads, still short of the chip: splits toward ~128
            // workgroups, and two key groups of two waves taking alternate tiles
            long ns = (128 + wgs / 2) / wgs;
            ns = ns < 1 ? 1 : (ns > kMaxSplit ? kMaxSplit : ns);
            c.ns = (int)ns;
            if ((ntiles + c.ns - 1) / c.ns >= 2) c.g = 2;
        }
    }
    c.tps = ntiles > 0 ? (ntiles + c.ns - 1) / c.ns : 1;
    c.ns = ntiles > 0 ? (ntiles + c.tps - 1) / c.tps : 1;   // no empty split
    return c;
}

using AttnKernel = void (*)(AttnArgs, int, int);

template <int DH, bool KV8>
AttnKernel attention_kernel(const AttnCfg& c) {
    // the fp8 cache's staging registers do not fit the two-group 4-wave
    // kernel (it would spill), so that shape runs one group with fp8
    if (c.g == 2 && c.waves == 2) return attn_mfma_kernel<DH, 2, 2, KV8>;
    if constexpr (!KV8)
        if (c.g == 2) return attn_mfma_kernel<DH, 4, 2, false>;
    return c.waves == 2 ? attn_mfma_kernel<DH, 2, 1, KV8> : attn_mfma_kernel<DH, 4, 1, KV8>;
}

}  // namespace

int attention_tiles(int masked, int P, int B, int nkeys) {
    return masked ? (P + kKeys - 1) / kKeys + (2 * B + kKeys - 1) / kKeys : (nkeys + kKeys - 1) / kKeys;
}

size_t attention_partial_slots(int dtype, int b, int R, int Hq, int Hkv, int ntiles) {
    if (dtype != DARD_DTYPE_BF16 || b < 1 || R < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv) return 0;
    const AttnCfg c = attention_cfg(b, R, Hq, Hkv, ntiles);
    return c.ns <= 1 ? 0 : (size_t)c.ns * b * R * Hq;
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
    if (a.out_frag && !frag_rows(dtype, a.b * a.R)) return hipErrorInvalidValue;
    if (a.Hkv < 1 || a.Hq % a.Hkv) return hipErrorInvalidValue;
    if (dtype == DARD_DTYPE_BF16) {
        if (a.masked && (!a.sel || a.B > kMaxBlock)) return hipErrorInvalidValue;
        if (a.dh != 64 && a.dh != 128) return hipErrorInvalidValue;
        const int ntiles = attention_tiles(a.masked, a.P, a.B, a.nkeys);
        AttnCfg c = attention_cfg(a.b, a.R, a.Hq, a.Hkv, ntiles);
        if (a.kv_fp8 && c.waves == 4) c.g = 1;   // see attention_kernel: one key group with the fp8 cache
        // a split needs room for its partials; without it one workgroup walks every key
        const size_t nrow = (size_t)a.b * a.R * a.Hq;
        if (c.ns > 1 && (!a.part || !a.part_ml || (size_t)c.ns * nrow > a.part_slots)) {
            c.ns = 1;
            c.tps = ntiles > 0 ? ntiles : 1;
        }
        const size_t tiles = (size_t)a.b * a.Hkv * c.rowtiles;
        if (tiles == 0 || tiles > 0x7fffffff) return hipErrorInvalidValue;
        dim3 grid((unsigned)tiles, c.ns);
        const AttnKernel k = a.kv_fp8 ? (a.dh == 128 ? attention_kernel<128, true>(c) : attention_kernel<64, true>(c))
                                      : (a.dh == 128 ? attention_kernel<128, false>(c) : attention_kernel<64, false>(c));
        launch(k, grid, dim3(64 * c.waves * c.g), 0, s, a, c.rowtiles, c.tps);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || c.ns == 1) return e;
        const size_t threads = nrow * (a.dh / 4);
        if (a.dh == 128)
            launch(attn_combine_kernel<128>, dim3((threads + 255) / 256), dim3(256), 0, s, a.part, a.part_ml, c.ns,
                   nrow, a.Hq, a.out_frag, reinterpret_cast<bf16_t*>(a.out));
        else
            launch(attn_combine_kernel<64>, dim3((threads + 255) / 256), dim3(256), 0, s, a.part, a.part_ml, c.ns,
                   nrow, a.Hq, a.out_frag, reinterpret_cast<bf16_t*>(a.out));
        return hipGetLastError();
    }
    if (a.kv_fp8) return hipErrorInvalidValue;   // the fp8 cache is a bf16-model variant
    const size_t total = (size_t)a.b * a.R * a.Hq;
    dim3 grid((total + 63) / 64);
    if (a.dh == 128)
        launch(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
    else
        launch(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
    return hipGetLastError();
}

}  // namespace dard
