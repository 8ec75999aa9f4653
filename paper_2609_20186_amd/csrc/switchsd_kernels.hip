// switchsd_kernels.hip -- gfx950 kernels of SwitchSD's speculation-control step.
//
// One kernel body (k_switchsd) serves the greedy step and its stages.  Its
// work-groups take one of three roles by block index, laid out as
// [probe | scan tiles | argmax segments, segment-major]:
//
//   scan    a 1024-position tile of one context, staged in LDS with a
//           64-token halo; ballots over blocks of 64 end positions mark the
//           occurrences of each suffix n-gram; the most recent end per n-gram
//           length is max-reduced over the work-group and (atomicMax) the
//           tiles of the sequence, and with W candidates each marked end is
//           written at its recency rank (the W most recent per wave and
//           length), merged latest wave and latest tile first.
//           (Sec. 3.3: kappa-gram with a prior occurrence, ranked by recency.)
//   probe   w . h for one sequence: exact bf16 x float products, summed in
//           double-double with a fixed reduction order.  (Sec. 3.2, Eq. 3.)
//   argmax  one segment of one logits row, streamed in 16 KB chunks with the
//           next chunk's nontemporal 16-byte loads in flight while the current
//           one is reduced.  Lane maxima of a chunk are packed 16-bit integer
//           maxima of the bf16 bit patterns (0.5 VALU ops per element), with
//           a float path for chunks holding a positive NaN or nothing >= +0;
//           each lane keeps the chunk that raised its maximum (in LDS) and
//           looks up the lowest index holding it once, at the end, before
//           one wave reduction.
//           The segment result is packed as (order key << 32 | ~index) and
//           stored in the segment's own slot (or atomicMax-ed into the row's
//           key).  (Sec. 2 / App. A: greedy verification, T = 0.)
//
// Two epilogues close a sequence without a second launch:
//   front   once its scan tiles and probe are done: pick the match, gather the
//           copy candidates, apply the switch (Sec. 3.3, Eq. 4) and write the
//           chosen draft (W candidates: W chains behind the anchor);
//   accept  once every row maximum is in: decode the row argmaxes and run the
//           accept walk (Sec. 3.3, Parallel Verification): a ballot for chains
//           and pointer jumping over trees, in registers (one node per lane)
//           up to 64 nodes and in LDS beyond.
// Where few enough work-groups wait (one per sequence, B no larger than the
// CU count), the hand-offs are polled: the last scan tile polls the other
// tiles' slots and runs the front, then, holding the draft, polls the argmax
// segments' slots and runs the accept epilogue; every other work-group stores
// its result and ends.  Otherwise the last work-group to arrive at a ticket
// runs the epilogue.  With the decode loop's commit the accept epilogue also
// appends the accepted tokens and the bonus to the context.  Each epilogue
// resets the workspace slots it consumed, leaving them zeroed for the next
// call.
//
// Further kernels: k_verify_poll (the greedy verify launch with polling),
// k_verify_stream (verification of long drafts over a fixed grid),
// k_sample_sums / k_sample_sums_stream and k_spec_residual (verification at
// sampling temperature T > 0), k_select and k_commit (stage entry points),
// k_tree_mask (the verification mask), k_label_insert / k_label_write /
// k_label_clear (copy-mode labels for probe training).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "switchsd_internal.h"

namespace switchsd {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = kThreads / 64;
constexpr int kScanBlocks = kScanTile / kThreads;  // blocks of 64 positions per scan wave
constexpr int kScanOffsets = 4;  // offsets u whose LDS reads are issued together
constexpr uint32_t kNoIdx = 0xFFFFFFFFu;

// Copy candidates being turned into a draft: end, length and first node of
// candidate c (W > 1).
struct ChainShared {
    int32_t e[kMaxCand];
    int32_t cl[kMaxCand];
    int32_t st[kMaxCand];
};
struct ScanShared {
    int32_t tile[kScanTile + 64];
    int32_t pat[SWITCHSD_MAX_NGRAM_LEN];
    int32_t red[SWITCHSD_MAX_NGRAM];
    // W > 1: each wave's W most recent ends + 1 per n-gram length, then the
    // work-group's merged list
    int32_t cand[SWITCHSD_MAX_NGRAM * kWaves * kMaxCand];
    int32_t merged[kMaxCand];
    ChainShared ch;
    // the neural draft, staged while the scan runs (general select path)
    int32_t nt[SWITCHSD_MAX_R];
    int32_t np[SWITCHSD_MAX_R];
    // the copy candidates' tokens, candidate c at c * k (general select path)
    int32_t ctok[SWITCHSD_MAX_R];
    double ps[kWaves];  // probe partial sums of the waves (scan tile 0)
    double pc[kWaves];
    int32_t L;
};
struct ArgmaxShared {
    float wmax[kWaves];
    uint32_t widx[kWaves];
    u32x4 keep[kChunkVecs];  // each lane's kept chunk (running argmax)
};
struct ProbeShared {
    double s[kWaves];
    double c[kWaves];
};
struct EpiShared {  // accept over R > 64 nodes
    int32_t a[SWITCHSD_MAX_R];
    int32_t tok[SWITCHSD_MAX_R];
    int32_t par[SWITCHSD_MAX_R];
    uint32_t st[2][SWITCHSD_MAX_R];  // pointer-jumping state, double-buffered (final_epilogue)
};
struct PickShared {  // one row's draw at T > 0
    unsigned long long cw[64 * kWaves];  // the row's weight sums per (chunk, wave)
    int32_t last;                      // this work-group completed the row (row_done)
};
struct PollShared {  // the segment results a sequence's accept epilogue polled
    unsigned long long k[kMaxSegs * 64];
};
struct DrawShared {  // one row's polled draw at T > 0 (draw_poller)
    unsigned long long cw[64 * kWaves];  // the row's weight sums per (chunk, wave)
    unsigned long long bs[kWaves];       // block sums of the chosen entry (wave w: block w)
    unsigned long long tg;               // the target within the entry
    unsigned long long key;              // the drawn token's key
    int32_t cst, est, ok;                // the entry (chunk, wave); every sum arrived
};
union Shared {
    ScanShared scan;
    PollShared poll;
    ArgmaxShared am;
    ProbeShared probe;
    EpiShared epi;
    PickShared pick;
    DrawShared draw;
};

// Timeline build only (compiled with SWITCHSD_TIMELINE, never in the product
// library): per work-group stamps of the 100 MHz real-time clock, slot
// [blk * 8 + i]: 0 start, 1 role done, 2 front done, 3 arrival done (with
// polling: every segment result seen), 4 epilogue done (its stores complete),
// 5 the epilogue's loads returned (with polling: the accept poll started),
// 6 poll rounds (accept poll << 32 | tile poll, each + 1),
// 7 = role << 32 | sequence.
#ifdef SWITCHSD_TIMELINE
#define TL_MARK(i)                                                                           \
    do {                                                                                     \
        if (threadIdx.x == 0 && p.tl)                                                        \
            p.tl[(int64_t)blockIdx.x * 8 + (i)] = __builtin_amdgcn_s_memrealtime();         \
    } while (0)
#define TL_TAG(v)                                                                            \
    do {                                                                                     \
        if (threadIdx.x == 0 && p.tl)                                                        \
            p.tl[(int64_t)blockIdx.x * 8 + 7] = (v);                                         \
    } while (0)
#define TL_ADD(i, v)                                                                         \
    do {                                                                                     \
        if (threadIdx.x == 0 && p.tl)                                                        \
            p.tl[(int64_t)blockIdx.x * 8 + (i)] += (v);                                      \
    } while (0)
#else
#define TL_MARK(i) \
    do {           \
    } while (0)
#define TL_TAG(v) \
    do {          \
    } while (0)
#define TL_ADD(i, v) \
    do {             \
    } while (0)
#endif

// ------------------------------------------------------------- atomics

__device__ __forceinline__ int32_t ld_i32(const int32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_i32(int32_t *p, int32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_f32(const float *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_f32(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_u64(const unsigned long long *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u64(unsigned long long *p, unsigned long long v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_u32(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u32(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wave 0 arrives at a per-sequence ticket; true (wave-uniform) for the last
// of `expected` arrivals.
//
// Every value one work-group hands to another travels through agent-scope
// atomics (RMW slots, or relaxed atomic stores and loads), which are coherent
// across the XCDs without any L2 write-back or invalidation.  Waiting for this
// wave's outstanding memory operations (vmcnt = 0) before the arrival
// therefore orders all of them ahead of it; the last arriver's reads are
// issued only after its arrival has returned.  An agent-scope release/acquire
// fence would give the same order but write back and invalidate the L2 of the
// XCD at every arrival, which costs more than the whole step.
__device__ __forceinline__ bool arrive(uint32_t *ticket, uint32_t expected) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0);
    uint32_t old = 0;
    if (threadIdx.x == 0)
        old = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    old = __shfl(old, 0);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    return old + 1u == expected;
}

// ------------------------------------------------------------- wave reductions (DPP)

// Row shifts 1, 2, 4, 8 give every lane the reduction of its 16-lane row up
// to itself; two row broadcasts fold the rows into lane 63.  Lanes whose DPP
// source is out of range keep the identity.
template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v, uint32_t id, Op op) {
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x111, 0xf, 0xf, false));
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x112, 0xf, 0xf, false));
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x114, 0xf, 0xf, false));
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x118, 0xf, 0xf, false));
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x142, 0xa, 0xf, false));
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x143, 0xc, 0xf, false));
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ float wave_max_f32(float v) {
    auto op = [](uint32_t a, uint32_t b) {
        return __float_as_uint(
            __builtin_elementwise_maximum(__uint_as_float(a), __uint_as_float(b)));
    };
    return __uint_as_float(wave_reduce_u32(__float_as_uint(v), 0xFF800000u, op));
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
    return wave_reduce_u32(v, 0xFFFFFFFFu, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    return wave_reduce_u32(v, 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

// ------------------------------------------------------------- probe role

__device__ __forceinline__ void two_sum(double a, double b, double &s, double &e) {
    s = a + b;
    const double bb = s - a;
    e = (a - (s - bb)) + (b - bb);
}
__device__ __forceinline__ void dd_add_term(double &s, double &c, double x) {
    double e;
    two_sum(s, x, s, e);
    c += e;
}
__device__ __forceinline__ void dd_add(double &s, double &c, double s2, double c2) {
    double e;
    two_sum(s, s2, s, e);
    c += c2 + e;
    double t;
    two_sum(s, c, t, c);  // renormalize
    s = t;
}
__device__ __forceinline__ double bf16_lo(uint32_t x) { return (double)__uint_as_float(x << 16); }
__device__ __forceinline__ double bf16_hi(uint32_t x) {
    return (double)__uint_as_float(x & 0xFFFF0000u);
}

// This lane's share of w . h for sequence b, as a double-double (s, c),
// reduced over the wave.  kGroups groups of 8 elements per lane (2048 kGroups
// elements per work-group) are requested before any is used: the stand-alone
// probe work-group takes 4 (all of d = 8192 in one memory round trip; its
// loads queue behind the argmax streams at 1-2 us per round trip), scan tile 0
// 2 (its scan state is live, and more would raise the kernel's registers).
template <int kGroups>
__device__ __forceinline__ void probe_partial(const StepParams &p, int b, double &s, double &c) {
    const int tid = threadIdx.x;
    const uint16_t *h = p.hidden + (int64_t)b * p.d;
    s = 0.0;
    c = 0.0;
    const bool vec = (p.d & 7) == 0 && (((uintptr_t)h | (uintptr_t)p.w) & 15) == 0;
    if (vec) {
        const u32x4 *hv = reinterpret_cast<const u32x4 *>(h);
        const float4 *wv = reinterpret_cast<const float4 *>(p.w);
        const int ng = p.d >> 3;
        for (int g0 = 0; g0 < ng; g0 += kGroups * kThreads) {
            u32x4 x[kGroups];
            float4 w0[kGroups], w1[kGroups];
#pragma unroll
            for (int q = 0; q < kGroups; ++q) {
                int g = g0 + q * kThreads + tid;
                g = g < ng ? g : ng - 1;
                x[q] = hv[g];
                w0[q] = wv[2 * g];
                w1[q] = wv[2 * g + 1];
            }
#pragma unroll
            for (int q = 0; q < kGroups; ++q) {
                if (g0 + q * kThreads + tid < ng) {
                    dd_add_term(s, c, bf16_lo(x[q][0]) * (double)w0[q].x);
                    dd_add_term(s, c, bf16_hi(x[q][0]) * (double)w0[q].y);
                    dd_add_term(s, c, bf16_lo(x[q][1]) * (double)w0[q].z);
                    dd_add_term(s, c, bf16_hi(x[q][1]) * (double)w0[q].w);
                    dd_add_term(s, c, bf16_lo(x[q][2]) * (double)w1[q].x);
                    dd_add_term(s, c, bf16_hi(x[q][2]) * (double)w1[q].y);
                    dd_add_term(s, c, bf16_lo(x[q][3]) * (double)w1[q].z);
                    dd_add_term(s, c, bf16_hi(x[q][3]) * (double)w1[q].w);
                }
            }
        }
    } else {
        for (int i = tid; i < p.d; i += kThreads)
            dd_add_term(s, c, bf16_lo((uint32_t)h[i]) * (double)p.w[i]);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const double s2 = __shfl_xor(s, o), c2 = __shfl_xor(c, o);
        dd_add(s, c, s2, c2);
    }
}

// Combines the waves' partial sums (fixed order) and the bias into z.
__device__ __forceinline__ float probe_combine(const double *ps, const double *pc, float bias) {
    double S = ps[0], C = pc[0];
    for (int q = 1; q < kWaves; ++q)
        dd_add(S, C, ps[q], pc[q]);
    dd_add(S, C, (double)bias, 0.0);
    return (float)(S + C);
}

// The chosen draft is written by the general path (LDS-staged neural draft,
// loops over nodes) rather than one node per lane of wave 0.
__device__ __forceinline__ bool general_select(const StepParams &p) {
    return p.W > 1 || p.R > 64 || p.k >= 64;
}

// The neural draft as handed over, read by wave 0 of a scan work-group before
// it is needed, so that the switch costs no extra round trip.
struct Prefetch {
    int nnb;   // node count clamped to [1, R]
    int ntok;  // ntok[b, lane] (lane < R <= 64)
    int npar;  // parent of node `lane`
};

// ------------------------------------------------------------- scan role

// Tile t of sequence b: end positions e in [t0, t0 + T) with T = kScanTile
// and t0 = t*T.  Leaves the tile's most recent end + 1 per n-gram length in
// sh.scan.red, the tokens of positions [t0 - 64, t0 + T) in sh.scan.tile
// (index = position - t0 + 64), with W > 1 the W most recent ends + 1 per
// length and wave in sh.scan.cand and, for tile 0 when the probe rides along,
// the waves' probe partial sums in sh.scan.ps/pc.
//
// Wave w owns the kScanBlocks blocks of 64 consecutive positions starting at
// t0 + w*T/4, one position per lane.  For suffix offset u, the ballot of
// (x[e-u] == x[L-1-u]) over a block marks its ends e whose u-th token back
// matches; AND-ing offsets 0..n-1 marks the ends of occurrences of the n-gram
// suffix, and the highest marked lane is the most recent one.  x[e-u] comes
// from the LDS tile (its 64-position halo covers u < 64), with the blocks'
// reads issued together: one compare and one 64-bit AND per block and offset.

// kMulti: the W > 1 candidate lists are compiled in (the host launches the
// instantiation that matches the configuration).
template <bool kMulti>
__device__ void scan_role(const StepParams &p, int b, int t, Shared &sh, Prefetch &pre) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int64_t row = (int64_t)b * p.Lmax;
    const int t0 = t * kScanTile;
    const int w0 = t0 + 64 * kScanBlocks * wave;  // first position of this wave

    // The tokens, the length, the suffix of a full-length context and the
    // neural draft do not depend on each other: issue all of them at once
    // (indices clamped into range, so that no load sits behind a branch).
    // tok[i + 1]: position w0 + 64 i + lane; tok[0]: the block before
    int32_t tok[kScanBlocks + 1];
#pragma unroll
    for (int i = 0; i <= kScanBlocks; ++i) {
        int x = w0 + 64 * (i - 1) + lane;
        x = x < 0 ? 0 : (x < p.Lmax ? x : p.Lmax - 1);
        tok[i] = p.tokens[row + x];
    }
    const int tp = tid < p.nmax ? tid : 0;
    const int32_t pat_full = p.tokens[row + (p.Lmax - 1 - tp >= 0 ? p.Lmax - 1 - tp : 0)];
    const int L = clampi(p.lengths[b], 0, p.Lmax);
    const bool stage_neural = p.epi_front == EPI_SELECT && general_select(p);
    int32_t snt[SWITCHSD_MAX_R / kThreads], snp[SWITCHSD_MAX_R / kThreads];
    if (p.epi_front == EPI_SELECT && tid < 64) {
        const int64_t base = (int64_t)b * p.R;
        const int i = tid < p.R ? tid : 0;
        pre.nnb = clampi(p.nn[b], 1, p.R);
        pre.ntok = p.ntok[base + i];
        pre.npar = p.npar ? p.npar[base + i] : tid - 1;
    }
    if (stage_neural) {
        const int64_t base = (int64_t)b * p.R;
#pragma unroll
        for (int q = 0; q < SWITCHSD_MAX_R / kThreads; ++q) {
            const int i = tid + kThreads * q;
            const int ic = i < p.R ? i : 0;
            snt[q] = p.ntok[base + ic];
            snp[q] = p.npar ? p.npar[base + ic] : i - 1;
        }
    }
    if (t == 0 && p.scan_probe) {
        double ps, pc;
        probe_partial<2>(p, b, ps, pc);
        if (lane == 0) {
            sh.scan.ps[wave] = ps;
            sh.scan.pc[wave] = pc;
        }
    }
    // the tile in LDS (for the copy candidate): index = position - t0 + 64
#pragma unroll
    for (int i = 0; i <= kScanBlocks; ++i)
        sh.scan.tile[64 * kScanBlocks * wave + 64 * i + lane] = tok[i];
    if (stage_neural) {
#pragma unroll
        for (int q = 0; q < SWITCHSD_MAX_R / kThreads; ++q)
            if (tid + kThreads * q < p.R) {
                sh.scan.nt[tid + kThreads * q] = snt[q];
                sh.scan.np[tid + kThreads * q] = snp[q];
            }
    }
    if (tid < SWITCHSD_MAX_NGRAM)
        sh.scan.red[tid] = 0;
    if (kMulti && p.W > 1)
        for (int i = tid; i < SWITCHSD_MAX_NGRAM * kWaves * kMaxCand; i += kThreads)
            sh.scan.cand[i] = 0;
    if (tid == 0)
        sh.scan.L = L;
    if (tid < p.nmax)
        sh.scan.pat[tid] = tid >= L ? 0 : (L == p.Lmax ? pat_full : p.tokens[row + L - 1 - tid]);
    __syncthreads();

    // bit n - 1 set for each configured length n; the lengths are strictly
    // descending, so length n is number popcount(bits above n - 1) in the list
    unsigned long long lenbits = 0ull;
#pragma unroll
    for (int j = 0; j < SWITCHSD_MAX_NGRAM; ++j)
        if (j < p.n_ngram)
            lenbits |= 1ull << (p.lens[j] - 1);
    int32_t best[SWITCHSD_MAX_NGRAM];
#pragma unroll
    for (int j = 0; j < SWITCHSD_MAX_NGRAM; ++j)
        best[j] = 0;
    // ends e <= L-2 of this wave's blocks
    const int elim = L - 1 - w0;  // e - w0 < elim
    if (elim > 0) {
        unsigned long long M[kScanBlocks];
#pragma unroll
        for (int i = 0; i < kScanBlocks; ++i) {
            const int n = elim - 64 * i;
            M[i] = n >= 64 ? ~0ull : (n <= 0 ? 0ull : ((1ull << n) - 1ull));
        }
        // LDS index of position w0 + 64 i + lane is lx0 + 64 i
        const int lx0 = w0 - t0 + 64 + lane;
        for (int u0 = 0; u0 < p.nmax; u0 += kScanOffsets) {
            // x[e - u] for kScanOffsets offsets u and every block: independent
            // LDS reads, issued together (one LDS wait per batch of offsets)
            int pu[kScanOffsets], xu[kScanOffsets][kScanBlocks];
#pragma unroll
            for (int du = 0; du < kScanOffsets; ++du) {
                const int u = u0 + du < p.nmax ? u0 + du : p.nmax - 1;
                pu[du] = sh.scan.pat[u];
#pragma unroll
                for (int i = 0; i < kScanBlocks; ++i)
                    xu[du][i] = u == 0 ? tok[i + 1] : sh.scan.tile[lx0 + 64 * i - u];
            }
#pragma unroll
            for (int du = 0; du < kScanOffsets; ++du) {
                const int u = u0 + du;
                if (u >= p.nmax)
                    break;
                // positions e < u have no u-th token back (only in the context's
                // first block)
#pragma unroll
                for (int i = 0; i < kScanBlocks; ++i)
                    M[i] &= __ballot(xu[du][i] == pu[du] && (i > 0 || w0 > 0 || lane >= u));
                // record the length equal to u + 1, if it is one of the lengths
                if ((lenbits >> u) & 1ull) {
                    const int jm = u == 63 ? 0 : __popcll(lenbits >> (u + 1));
                    int e1 = 0;
#pragma unroll
                    for (int i = 0; i < kScanBlocks; ++i)
                        if (M[i])
                            e1 = w0 + 64 * i + 64 - __clzll((long long)M[i]);  // highest end + 1
#pragma unroll
                    for (int j = 0; j < SWITCHSD_MAX_NGRAM; ++j)
                        if (j == jm)
                            best[j] = e1;
                    if (kMulti && p.W > 1) {
                        // this wave's W most recent ends of this length: each
                        // lane writes its own end at its rank among the ends
                        // at later positions (later blocks, then higher lanes)
                        int32_t *dst = &sh.scan.cand[(jm * kWaves + wave) * kMaxCand];
                        int later = 0;
#pragma unroll
                        for (int i = kScanBlocks - 1; i >= 0; --i) {
                            const unsigned long long above =
                                lane == 63 ? 0ull : (M[i] >> (lane + 1));
                            const int rank = later + __popcll(above);
                            if (((M[i] >> lane) & 1ull) && rank < p.W)
                                dst[rank] = w0 + 64 * i + lane + 1;
                            later += __popcll(M[i]);
                        }
                    }
                }
            }
        }
    }
#pragma unroll
    for (int j = 0; j < SWITCHSD_MAX_NGRAM; ++j)
        if (j < p.n_ngram && lane == 0 && best[j] > 0)
            atomicMax(&sh.scan.red[j], best[j]);
    __syncthreads();
}

// In the step with several scan tiles per sequence the probe has a
// work-group of its own, dispatched before every tile (block order), and the
// tile that chooses the draft waits for this flag before it reads z.  It sits
// in the last word of the sequence's n-gram slot line (at most 8 n-gram
// lengths use the line).  (Measured: z and a ready bit in one 64-bit word,
// read once, made C3 and C4 0.05-0.1 us slower than the flag and a second
// read.)
__device__ __forceinline__ uint32_t *probe_flag(const StepParams &p, int b) {
    return (uint32_t *)&p.ws.mslot[b * kLineU32 + kLineU32 - 1];
}

// Device-side error word of sequence b, next to the probe flag: nonzero when
// a bounded wait of this call gave up (read and cleared by
// switchsd_workspace_status).
__device__ __forceinline__ uint32_t *error_word(const StepParams &p, int b) {
    return (uint32_t *)&p.ws.mslot[b * kLineU32 + kLineU32 - 2];
}

// Stand-alone probe work-group (the probe entry point, or the step's probe
// when a sequence has several scan tiles).
__device__ void probe_role(const StepParams &p, int b, Shared &sh) {
    double s, c;
    probe_partial<4>(p, b, s, c);
    const int tid = threadIdx.x;
    if ((tid & 63) == 0) {
        sh.probe.s[tid >> 6] = s;
        sh.probe.c[tid >> 6] = c;
    }
    __syncthreads();
    if (tid == 0) {
        st_f32(&p.z[b], probe_combine(sh.probe.s, sh.probe.c, p.bias));
        if (p.epi_front == EPI_SELECT && !p.withhold_flag) {  // the step: z is ready
            __builtin_amdgcn_s_waitcnt(0);
            st_u32(probe_flag(p, b), 1u);
        }
    }
}

// ------------------------------------------------------------- argmax role

__device__ __forceinline__ float lo_f(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float hi_f(uint32_t x) { return __uint_as_float(x & 0xFFFF0000u); }
__device__ __forceinline__ float max3n(float a, float b, float c) {
    return __builtin_elementwise_maximum(a, __builtin_elementwise_maximum(b, c));
}

// Order-preserving key of a float; -0 is folded onto +0.
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Sequence b is verified by speculative sampling with its draft's own
// distribution q (T > 0): q is given and the chosen draft is the neural one.
__device__ __forceinline__ bool spec_seq(const StepParams &p, int b) {
    return p.qlogits != nullptr && !(p.spec_copy && ld_i32(&p.spec_copy[b]) != 0);
}

// Rows a sequence may need, as rows_needed with the node count already read:
// every row; the chosen draft's nnb nodes (verify launch); or the longer of
// the neural draft (nnb nodes) and the longest copy draft (fused step).
__device__ __forceinline__ uint32_t rows_of_drafts(const StepParams &p, int nnb) {
    if (p.rows_mode == ROWS_ALL)
        return (uint32_t)p.R;
    if (p.rows_mode == ROWS_DRAFT)
        return (uint32_t)nnb;
    const int cn = 1 + p.W * p.k;  // the longest copy draft
    return (uint32_t)(nnb > cn ? nnb : cn);
}

__device__ __forceinline__ uint32_t rows_needed(const StepParams &p, int b) {
    if (p.rows_mode == ROWS_ALL || p.rows_mode == ROWS_LISTED)
        return (uint32_t)p.R;
    if (p.rows_mode == ROWS_DRAFT)
        return (uint32_t)clampi(ld_i32(&p.dn[b]), 1, p.R);
    if (p.rows_mode == ROWS_Q)  // q at the rows that have a drafted child
        return spec_seq(p, b) ? (uint32_t)(clampi(ld_i32(&p.dn[b]), 1, p.R) - 1) : 0u;
    return rows_of_drafts(p, clampi(p.nn[b], 1, p.R));
}

// Running argmax of one lane over the 16 KB chunks it reduces, in increasing
// index order.  Per chunk only the lane's maximum is taken; the chunk that
// raised it is kept, and the lowest index holding the maximum is looked up
// once at the end (lazy_index), so the streaming loop carries no cross-lane
// work.  best is NaN while the lane has seen no non-NaN element.  The kept
// chunk sits in registers (LazyMax) or, where registers are short, in LDS
// (LazyMaxLds: vector u of lane t at d[u * kThreads + t]).
struct LazyMax {
    float best;
    int q0;                 // first vector index of the kept chunk
    u32x4 d[kUnroll];       // the kept chunk
    __device__ __forceinline__ u32x4 get(int u) const { return d[u]; }
    __device__ __forceinline__ void keep(bool upd, const u32x4 (&v)[kUnroll]) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int w4 = 0; w4 < 4; ++w4)
                d[u][w4] = upd ? v[u][w4] : d[u][w4];
    }
};
struct LazyMaxLds {
    float best;
    int q0;
    u32x4 *d;
    __device__ __forceinline__ u32x4 get(int u) const { return d[u * kThreads + threadIdx.x]; }
    __device__ __forceinline__ void keep(bool upd, const u32x4 (&v)[kUnroll]) {
        if (upd) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                d[u * kThreads + threadIdx.x] = v[u];
        }
    }
};

template <typename S>
__device__ __forceinline__ void lazy_init(S &s) {
    s.best = __builtin_nanf("");
    s.q0 = 0;
}

// Maximum ignoring NaN; NaN only when both are NaN (or m is and x is).
__device__ __forceinline__ float fmax_first(float m, float x) {
    return (m != m || x > m) ? x : m;
}

typedef short s16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ s16x2 as_s16x2(uint32_t u) { return __builtin_bit_cast(s16x2, u); }

// Maximum of the 8 * kUnroll elements of a lane's chunk as floats, NaN ignored
// (NaN only when every element is NaN).
__device__ __forceinline__ float chunk_max(const u32x4 (&v)[kUnroll]) {
    float m = -__builtin_inff();
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        m = max3n(m, lo_f(v[u][0]), hi_f(v[u][0]));
        m = max3n(m, lo_f(v[u][1]), hi_f(v[u][1]));
        m = max3n(m, lo_f(v[u][2]), hi_f(v[u][2]));
        m = max3n(m, lo_f(v[u][3]), hi_f(v[u][3]));
    }
    if (m != m) {  // a NaN somewhere: recompute ignoring NaN
        m = __builtin_nanf("");
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int w4 = 0; w4 < 4; ++w4) {
                m = fmax_first(m, lo_f(v[u][w4]));
                m = fmax_first(m, hi_f(v[u][w4]));
            }
    }
    return m;
}

// Chunk [qc0, qc0 + kChunkVecs) of a row piece of nq vectors; vectors past nq
// read as -inf and are never reported (lazy_index checks q < nq).  A later
// chunk replaces the kept one only with a strictly larger maximum, so ties
// stay with the earliest chunk.
template <typename S>
__device__ __forceinline__ void lazy_chunk(u32x4 (&v)[kUnroll], int qc0, int nq, S &s) {
    const int tid = threadIdx.x;
    if (qc0 + kChunkVecs > nq) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (qc0 + u * kThreads + tid >= nq)
                v[u] = u32x4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};
    }
    // Read as signed 16-bit integers, the bf16 bit patterns of +0 .. +inf keep
    // their order and sit above every negative pattern, and positive NaNs sit
    // above +inf; one packed integer maximum per two elements then gives the
    // chunk's maximum whenever it lies in [+0, +inf].  Otherwise (a positive
    // NaN, or no element >= +0) the floats are compared, unless the lane
    // already holds a maximum >= +0 that an all-negative chunk cannot raise.
    static_assert(kUnroll == 4, "the packed maximum below takes four vectors per lane");
    s16x2 t[4];
#pragma unroll
    for (int w4 = 0; w4 < 4; ++w4)
        t[w4] = __builtin_elementwise_max(
            __builtin_elementwise_max(as_s16x2(v[0][w4]), as_s16x2(v[1][w4])),
            __builtin_elementwise_max(as_s16x2(v[2][w4]), as_s16x2(v[3][w4])));
    t[0] = __builtin_elementwise_max(__builtin_elementwise_max(t[0], t[1]),
                                     __builtin_elementwise_max(t[2], t[3]));
    const int m16 = t[0].x > t[0].y ? t[0].x : t[0].y;
    float m = m16 >= 0 ? __uint_as_float((uint32_t)m16 << 16) : -__builtin_inff();
    const bool exact = m16 > 0x7F80 || (m16 < 0 && !(s.best >= 0.0f));
    if (__any(exact)) {
        if (exact)
            m = chunk_max(v);
    }
    const bool upd = m == m && !(m <= s.best);
    s.best = upd ? m : s.best;
    s.q0 = upd ? qc0 : s.q0;
    s.keep(upd, v);
}

// Lowest row-relative index (vector q is at ebase + 8q) of an element equal to
// the lane's maximum in its kept chunk; kNoIdx when the lane has none.  -0 and
// +0 compare equal.
template <typename S>
__device__ __forceinline__ uint32_t lazy_index(const S &s, int nq, uint32_t ebase) {
    uint32_t idx = kNoIdx;
    if (s.best == s.best) {
#pragma unroll
        for (int u = kUnroll - 1; u >= 0; --u) {  // descending: the last hit is the lowest
            const int q = s.q0 + u * kThreads + (int)threadIdx.x;
            const uint32_t e = ebase + (uint32_t)q * 8u;
            const u32x4 d = s.get(u);
#pragma unroll
            for (int w4 = 3; w4 >= 0; --w4) {
                if (q < nq && hi_f(d[w4]) == s.best)
                    idx = e + w4 * 2u + 1u;
                if (q < nq && lo_f(d[w4]) == s.best)
                    idx = e + w4 * 2u;
            }
        }
    }
    return idx;
}

// Wave argmax of (value, index) pairs, index kNoIdx meaning none: the largest
// value, ties to the lowest index.  Returns the index (kNoIdx when the wave has
// none) and the value in W.
__device__ __forceinline__ uint32_t wave_argmax(float v, uint32_t idx, float &W) {
    W = wave_max_f32(idx != kNoIdx ? v : -__builtin_inff());
    return wave_min_u32(idx != kNoIdx && v == W ? idx : kNoIdx);
}

__device__ __forceinline__ void load_chunk(u32x4 (&v)[kUnroll], const u32x4 *vp, int qc0, int nq) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int q = qc0 + u * kThreads + (int)threadIdx.x;
        v[u] = __builtin_nontemporal_load(vp + (q < nq ? q : nq - 1));
    }
}

// Segment s of row r of sequence b.
// qpart: a segment of the draft's logits (row maxima of q, into the q keys)
// in a row maxima launch that takes the q rows too.
__device__ __forceinline__ uint32_t q_rows(const StepParams &p, int b) {
    // with the front in the same launch the draft is not chosen yet: the rows
    // of the neural draft that have a drafted child (a copy draft's q is
    // one-hot and needs none); else the rows with a drafted child of the
    // sequences verified with q
    if (p.epi_front == EPI_SELECT)
        return (uint32_t)(clampi(p.nn[b], 1, p.R) - 1);
    return spec_seq(p, b) ? (uint32_t)(clampi(ld_i32(&p.dn[b]), 1, p.R) - 1) : 0u;
}

__device__ void argmax_role(const StepParams &p, int b, int r, int s, Shared &sh, u32x4 *keep,
                            bool qpart = false) {
    const int tid = threadIdx.x;
    const uint16_t *lg = qpart ? p.qlogits : p.logits;
    const int64_t rowoff = ((int64_t)b * p.R + r) * p.V;
    const int64_t e0 = (int64_t)s * p.seg_elems;
    const int64_t e1 = e0 + p.seg_elems < p.V ? e0 + p.seg_elems : (int64_t)p.V;
    // element g of the tensor sits at byte 2g from the base: the 16-byte
    // aligned interior [a0, a1) is read with 16-byte loads, the head [g0, a0)
    // and the tail [a1, g1) (at most 7 elements each) one element per lane.
    const int64_t g0 = rowoff + e0, g1 = rowoff + e1;
    const int64_t mis = (int64_t)((((uintptr_t)lg) >> 1) + (uint64_t)g0) & 7;
    int64_t a0 = g0 + ((8 - mis) & 7);
    if (a0 > g1)
        a0 = g1;
    const int64_t a1 = a0 + ((g1 - a0) & ~(int64_t)7);
    const int nq = (int)((a1 - a0) >> 3);
    const u32x4 *vp = reinterpret_cast<const u32x4 *>(lg + a0);
    const uint32_t ebase = (uint32_t)(a0 - rowoff);

    const int nhead = (int)(a0 - g0), ntail = (int)(g1 - a1);
    int64_t xg = -1;
    if (tid < nhead)
        xg = g0 + tid;
    else if (tid < nhead + ntail)
        xg = a1 + (tid - nhead);
    const float xv = xg >= 0 ? lo_f((uint32_t)lg[xg]) : -__builtin_inff();
    const uint32_t xi = (uint32_t)(xg - rowoff);
    const bool has_x = xg >= 0;

    if (p.csum_clear && !qpart) {
        // this segment's share of the row's weight-sum slots, zeroed for the
        // pollers of the sum launch that follows (the polled draw at T > 0)
        const int n = p.cpr * kCsumPerChunk;
        const int i0 = s * n / p.segs, i1 = (s + 1) * n / p.segs;
        if (tid < i1 - i0)
            p.csum[((int64_t)b * p.R + r) * n + i0 + tid] = 0ull;
    }
    LazyMaxLds st;
    st.d = keep;
    lazy_init(st);
    const int nch = (nq + kChunkVecs - 1) / kChunkVecs;
    // Whether the row is needed at all may depend on the draft (a global read);
    // with `speculate` the first chunk is already in flight meanwhile.
    u32x4 A[kUnroll], Bv[kUnroll];
    const bool spec = p.speculate && nch > 0;
    if (spec)
        load_chunk(A, vp, 0, nq);
    if ((uint32_t)r >= (qpart ? q_rows(p, b) : rows_needed(p, b))) {
        __builtin_amdgcn_s_waitcnt(0);
        return;
    }
    if (nch > 0) {
        // double buffer: chunk c + 1 is in flight while chunk c is reduced.
        // The loop body has a single exit at its end, so that no path reaches
        // the next iteration with the other buffer's loads still pending (the
        // compiler would then wait for every load at the top of the loop).
        // A load past the last chunk reads the last vector again (clamped).
        if (!spec)
            load_chunk(A, vp, 0, nq);
        int c = 0;
        for (; c + 1 < nch; c += 2) {
            load_chunk(Bv, vp, (c + 1) * kChunkVecs, nq);
            lazy_chunk(A, c * kChunkVecs, nq, st);
            load_chunk(A, vp, (c + 2) * kChunkVecs, nq);
            lazy_chunk(Bv, (c + 1) * kChunkVecs, nq, st);
        }
        if (c < nch)  // odd count: the last chunk
            lazy_chunk(A, c * kChunkVecs, nq, st);
    }
    // the head and tail elements (lower and higher indices than the interior)
    float lv = st.best;
    uint32_t li = lazy_index(st, nq, ebase);
    if (has_x && xv == xv && (li == kNoIdx || xv > lv || (xv == lv && xi < li))) {
        lv = xv;
        li = xi;
    }
    float runM;
    const uint32_t runI = wave_argmax(lv, li, runM);
    const int wave = tid >> 6, lane = tid & 63;
    if (lane == 0) {
        sh.am.wmax[wave] = runM;
        sh.am.widx[wave] = runI;
    }
    __syncthreads();
    if (tid == 0) {
        float M = -__builtin_inff();
        uint32_t best = kNoIdx;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) {
            const uint32_t iq = sh.am.widx[q];
            const float mq = sh.am.wmax[q];
            if (iq != kNoIdx && (best == kNoIdx || mq > M || (mq == M && iq < best))) {
                M = mq;
                best = iq;
            }
        }
        const unsigned long long key =
            best != kNoIdx ? ((unsigned long long)order_key(M) << 32) | (0xFFFFFFFFu - best)
                           : 0ull;
        if (qpart) {
            if (key)
                atomicMax(&p.ws.qkeys[(int64_t)b * p.ws.key_stride + r], key);
        } else if (p.poll_accept) {
            // the segment's own slot (1: no candidate); nothing waits for the
            // store here, the sequence's epilogue polls for it
            if (!(p.withhold_seg && b == 0 && r == 0 && s == 0))
                st_u64(&p.ws.skeys[(int64_t)b * p.ws.skey_stride + (int64_t)s * p.R + r],
                       key ? key : 1ull);
        } else if (key) {
            atomicMax(&p.ws.keys[(int64_t)b * p.ws.key_stride + r], key);
        }
    }
}

// ------------------------------------------------------------- epilogues

// The chosen draft of a sequence as wave 0 of its front holds it (R <= 64):
// lane i has node i's token and parent (-1 past the draft), every lane the
// node count, the switch decision and the neural draft's clamped node count
// (set where the neural draft was read, so that no later use waits for that
// read again).  With `deferred` the front's outputs are not written yet: the
// match (mn, me, cl; lane j < k holds copied token ct), the draft, the score z
// when this work-group computed it (zstore), the clearing of the probe's flag
// (zclear) and of the tile slots this lane polled (bit q of tclear: slot
// q * 64 + lane) go out with store_front once the accept epilogue has polled
// its results, so that its first poll does not also wait for these stores
// (a wave's loads and stores complete in one count).
struct DraftRegs {
    int tok, par, dn, use, nnb;
    int mn, me, cl, ct;
    float z;
    uint32_t tclear;
    bool deferred, zstore, zclear;
};

__device__ __forceinline__ uint32_t *probe_flag(const StepParams &p, int b);

// Outputs of steps 1 and 3 from dr (wave 0; one candidate, R <= 64, k < 64).
__device__ void store_front(const StepParams &p, int b, const DraftRegs &dr, bool select) {
    const int lane = threadIdx.x;
    const int64_t base = (int64_t)b * p.R;
    if (lane == 0) {
        p.match_n[b] = dr.mn;
        p.match_end[b] = dr.me;
        p.copy_len[b] = dr.cl;
        if (dr.zstore)
            p.z[b] = dr.z;
        if (dr.zclear)
            st_u32(probe_flag(p, b), 0u);
    }
    if (dr.tclear) {
        int32_t *ts = p.ws.tslot + (int64_t)b * p.ws.tslot_stride;
        for (int q = 0; q < 8; ++q)
            if ((dr.tclear >> q) & 1u)
                st_i32(&ts[q * 64 + lane], 0);
    }
    if (lane < p.k)
        p.copy_tokens[(int64_t)b * p.k + lane] = dr.ct;
    if (select) {
        if (lane < p.R) {
            st_i32(&p.dtok[base + lane], dr.tok);  // read by the accept epilogue of this launch
            st_i32(&p.dpar[base + lane], dr.par);
        }
        if (lane == 0) {
            st_i32(&p.use_copy[b], dr.use);  // read by the commit of this launch
            st_i32(&p.dn[b], dr.dn);
        }
    }
}

// Steps 1 and 3 for sequence b in wave 0 once the match (mn, me) is known:
// copy candidate, switch (Eq. 4 with the kappa gate), chosen draft (also left
// in dr).  When `have_ct`, ct_in is this lane's copied token (read from LDS
// by the caller); otherwise it is read from the context here.
__device__ void front_finish(const StepParams &p, int b, int mn, int me, int L, float zb,
                             const Prefetch &pre, int ct_in, bool have_ct, DraftRegs &dr) {
    const int lane = threadIdx.x;
    const int64_t row = (int64_t)b * p.Lmax;
    const bool select = p.epi_front == EPI_SELECT;
    const int cl = mn > 0 ? (p.k < L - 1 - me ? p.k : L - 1 - me) : 0;
    // lane j holds copied token j (R <= 64, k < 64, one candidate)
    const int ct = lane < cl ? (have_ct ? ct_in : p.tokens[row + me + 1 + lane]) : -1;
    dr.mn = mn;
    dr.me = me;
    dr.cl = cl;
    dr.ct = ct;
    dr.deferred = select && p.poll_accept;
    if (select) {
        const int use = (mn >= p.kappa) && (zb >= p.theta);
        const int dnb = use ? cl + 1 : pre.nnb;
        const int ctp = __shfl(ct, lane >= 1 ? lane - 1 : 0);
        int tok = -1, par = -1;
        if (lane >= 1 && lane < dnb) {
            tok = use ? ctp : pre.ntok;
            par = use ? lane - 1 : pre.npar;
        }
        dr.tok = tok;
        dr.par = par;
        dr.dn = dnb;
        dr.use = use;
        dr.nnb = pre.nnb;
    }
    if (!dr.deferred)
        store_front(p, b, dr, select);
}

// First length (in the configured order) whose slot holds an occurrence:
// (match_n, match_end, its index jsel), or (0, -1, -1).  s is lane j's slot
// value (end + 1).
__device__ __forceinline__ void pick_match(const StepParams &p, int32_t s, int &mn, int &me,
                                           int &jsel) {
    const unsigned long long hit = __ballot(s > 0);
    mn = 0;
    me = -1;
    jsel = -1;
    if (hit) {
        const int j = __ffsll((long long)hit) - 1;
        jsel = j;
#pragma unroll
        for (int q = 0; q < SWITCHSD_MAX_NGRAM; ++q)
            if (q == j)
                mn = p.lens[q];
        me = __shfl(s, j) - 1;
    }
}

// ------------------------------------------------------------- W > 1 copy candidates

// Wave 0: the work-group's W most recent ends + 1 of n-gram length j, merged
// over its four waves (a higher wave holds later positions).  Lane c < W
// receives the c-th, 0 past the last occurrence.
__device__ int merge_waves(const StepParams &p, Shared &sh, int j) {
    const int lane = threadIdx.x;
    const int W = p.W;
    int v = 0;
    if (lane < kWaves * W) {
        const int q = lane / W;
        v = sh.scan.cand[(j * kWaves + (kWaves - 1 - q)) * kMaxCand + (lane - q * W)];
    }
    if (lane < W)
        sh.scan.merged[lane] = 0;
    const unsigned long long nz = __ballot(v > 0);
    const int rank = __popcll(nz & ((1ull << lane) - 1ull));
    if (v > 0 && rank < W)
        sh.scan.merged[rank] = v;
    return lane < W ? sh.scan.merged[lane] : 0;
}

// Wave 0: lays W candidates of lengths cl (lane c) out as chains behind the
// anchor: ch.cl[c] and ch.st[c] (first node of candidate c).  Returns the node
// count 1 + sum of the lengths.
__device__ int chain_layout(const StepParams &p, int cl, ChainShared &ch) {
    const int lane = threadIdx.x;
    int inc = cl;  // inclusive prefix sum over lanes 0..W-1 (W <= 16)
#pragma unroll
    for (int o = 1; o < kMaxCand; o <<= 1) {
        const int y = __shfl_up(inc, o);
        if (lane >= o)
            inc += y;
    }
    if (lane < p.W) {
        ch.cl[lane] = cl;
        ch.st[lane] = 1 + inc - cl;
    }
    return 1 + __shfl(inc, p.W - 1);
}

// Wave 0: writes the chosen draft of sequence b (Eq. 4 with the kappa gate);
// a copy draft is the chains laid out in ch, token j of candidate c being
// src(c, j); the neural draft has nnb nodes, node i given by nsrc(i, tok, par).
// Nodes 0..63 are also left in dr.
template <typename Src, typename NSrc>
__device__ void write_chains(const StepParams &p, int b, int use, int total, int nnb,
                             const ChainShared &ch, Src src, NSrc nsrc, DraftRegs &dr) {
    const int lane = threadIdx.x;
    const int64_t base = (int64_t)b * p.R;
    const int dnb = use ? total : nnb;
    // the chains' first nodes in registers (one LDS read each, all at once)
    int stq[kMaxCand];
#pragma unroll
    for (int q = 0; q < kMaxCand; ++q)
        stq[q] = q < p.W ? ch.st[q] : 0x7FFFFFFF;
    dr = DraftRegs{-1, -1, dnb, use, nnb, 0, -1, 0, -1, 0.0f, 0u, false, false, false};
    for (int i = lane; i < p.R; i += 64) {
        int tok = -1, par = -1;
        if (i >= 1 && i < dnb) {
            if (use) {
                int c = 0, st = stq[0];  // the last chain starting at or before i
#pragma unroll
                for (int q = 1; q < kMaxCand; ++q)
                    if (stq[q] <= i) {
                        c = q;
                        st = stq[q];
                    }
                tok = src(c, i - st);
                par = i == st ? 0 : i - 1;
            } else {
                nsrc(i, tok, par);
            }
        }
        st_i32(&p.dtok[base + i], tok);  // read by the accept epilogue of the same launch
        st_i32(&p.dpar[base + i], par);
        if (i == lane) {
            dr.tok = tok;
            dr.par = par;
        }
    }
    if (lane == 0) {
        st_i32(&p.use_copy[b], use);  // read by the commit of this launch
        st_i32(&p.dn[b], dnb);
    }
}

// Steps 1 and 3 on the general path (wave 0 of a scan work-group).  Lane
// c < W holds v = end + 1 of candidate c (0: none).  Context positions in
// [lo, hi) are read from this work-group's LDS tile (index = position - t0 +
// 64), the others from memory; the neural draft was staged in LDS.
__device__ void front_finish_w(const StepParams &p, int b, int mn, int v, int L, float zb,
                               const Prefetch &pre, Shared &sh, int t0, int lo, int hi,
                               DraftRegs &dr) {
    const int lane = threadIdx.x;
    const int W = p.W;
    const int64_t row = (int64_t)b * p.Lmax;
    const int cl = (lane < W && v > 0) ? (p.k < L - v ? p.k : L - v) : 0;
    ChainShared &ch = sh.scan.ch;
    if (lane < W) {
        ch.e[lane] = v - 1;
        p.match_end[(int64_t)b * W + lane] = v - 1;
        p.copy_len[(int64_t)b * W + lane] = cl;
    }
    if (lane == 0)
        p.match_n[b] = mn;
    const int total = chain_layout(p, cl, ch);
    // every candidate's tokens into LDS, four per lane requested together (from
    // the LDS tile where they lie in it), then the outputs and the chains from
    // there: one memory round trip for W * k tokens
    const int ntk = W * p.k;
    for (int i0 = 0; i0 < ntk; i0 += 4 * 64) {
        int v4[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int idx = i0 + q * 64 + lane;
            const int c = idx < ntk ? idx / p.k : 0, j = idx - c * p.k;
            v4[q] = -1;
            if (idx < ntk && j < ch.cl[c]) {
                const int pos = ch.e[c] + 1 + j;
                v4[q] = (pos >= lo && pos < hi) ? sh.scan.tile[pos - t0 + 64]
                                                : ld_i32(&p.tokens[row + pos]);  // as in front_remote
            }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (i0 + q * 64 + lane < ntk)
                sh.scan.ctok[i0 + q * 64 + lane] = v4[q];
    }
    __builtin_amdgcn_wave_barrier();
    auto src = [&](int c, int j) -> int { return sh.scan.ctok[c * p.k + j]; };
    const int64_t cbase = (int64_t)b * W * p.k;
    for (int idx = lane; idx < ntk; idx += 64)
        p.copy_tokens[cbase + idx] = sh.scan.ctok[idx];
    if (p.epi_front == EPI_SELECT)
        write_chains(p, b, (mn >= p.kappa) && (zb >= p.theta), total, pre.nnb, ch, src,
                     [&](int i, int &tok, int &par) {
                         tok = sh.scan.nt[i];
                         par = sh.scan.np[i];
                     },
                     dr);
}

// A context held by one scan tile: everything the switch needs is already in
// this work-group (match in LDS, probe partial sums in LDS, the copy
// candidate in the LDS tile, the neural draft prefetched).  No arrival.
__device__ void front_local(const StepParams &p, int b, Shared &sh, const Prefetch &pre,
                            DraftRegs &dr) {
    const int lane = threadIdx.x;
    const int32_t s = lane < p.n_ngram ? sh.scan.red[lane] : 0;
    int mn, me, jsel;
    pick_match(p, s, mn, me, jsel);
    const int L = sh.scan.L;
    float zb = 0.0f;
    const bool defer = p.epi_front == EPI_SELECT && p.poll_accept && !general_select(p);
    if (p.scan_probe) {
        float z0 = 0.0f;
        if (lane == 0) {
            z0 = probe_combine(sh.scan.ps, sh.scan.pc, p.bias);
            if (!defer)
                p.z[b] = z0;
        }
        zb = __shfl(z0, 0);
        dr.z = zb;
        dr.zstore = defer;
    }
    if (general_select(p)) {
        const int v = mn <= 0 ? 0 : (p.W > 1 ? merge_waves(p, sh, jsel) : (lane == 0 ? me + 1 : 0));
        front_finish_w(p, b, mn, v, L, zb, pre, sh, 0, 0,
                       p.Lmax < kScanTile ? p.Lmax : kScanTile, dr);
        return;
    }
    const int pos = me + 1 + lane;  // tile index = position + 64 (tile 0)
    const int ct = (mn > 0 && lane < p.k && pos < L) ? sh.scan.tile[pos + 64] : -1;
    front_finish(p, b, mn, me, L, zb, pre, ct, true, dr);
}

// The scan tile that chooses the draft of a longer context, once every tile's
// result is in: s is lane j's n-gram slot value over all tiles (end + 1 of
// the most recent occurrence of length j, 0 none), fl0 a first read of the
// probe's flag (the step).  The copy candidate comes from this tile's LDS
// when it lies there, else from the context.
__device__ void front_remote(const StepParams &p, int b, int t, Shared &sh, const Prefetch &pre,
                             DraftRegs &dr, int32_t s, uint32_t fl0) {
    const int lane = threadIdx.x;
    int mn, me, jsel;
    pick_match(p, s, mn, me, jsel);
    const int L = sh.scan.L;
    // one candidate: its tokens are requested before the wait for the probe
    // (they do not depend on z), from this tile's LDS where they lie in it
    // (positions [t0 - 64, t0 + T), index = position - t0 + 64)
    const int t0 = t * kScanTile;
    int cl1 = 0, ct1 = -1;
    bool in_tile = false;
    if (!general_select(p)) {
        cl1 = mn > 0 ? (p.k < L - 1 - me ? p.k : L - 1 - me) : 0;
        const int lo = t0 - 64 > 0 ? t0 - 64 : 0;
        const int hi = t0 + kScanTile < p.Lmax ? t0 + kScanTile : p.Lmax;
        in_tile = cl1 > 0 && me + 1 >= lo && me + cl1 < hi;
        // (the context read is an atomic one, so that the compiler cannot
        // merge the two reads into one through a generic pointer: such a
        // read is counted as both an LDS and a memory access, and every
        // later wait for it would also wait for all of this wave's stores)
        if (lane < cl1)
            ct1 = in_tile ? sh.scan.tile[me + 1 + lane - t0 + 64]
                          : ld_i32(&p.tokens[(int64_t)b * p.Lmax + me + 1 + lane]);
    }
    float zb = 0.0f;
    if (p.epi_front == EPI_SELECT) {
        if (p.probe_on) {
            // the probe's work-group was dispatched before every tile and
            // depends on nothing, so the flag is set in bounded time; the cap
            // only guards against a broken launch.  If it is reached, the
            // sequence's error word is set and the switch takes the neural
            // draft (a NaN score never clears the threshold).
            uint32_t *fl = probe_flag(p, b);
            bool seen = __builtin_amdgcn_readfirstlane((int)fl0) != 0;
            for (int spin = 0; spin < p.spin_cap && !seen; ++spin) {
                __builtin_amdgcn_s_sleep(2);
                seen = __builtin_amdgcn_readfirstlane((int)ld_u32(fl)) != 0;
            }
            if (seen) {
                zb = ld_f32(&p.z[b]);
            } else {
                zb = __builtin_nanf("");
                if (lane == 0)
                    st_u32(error_word(p, b), 1u);
            }
            // with the accept epilogue polling, the clearing goes out after its
            // poll (store_front)
            dr.zclear = p.poll_accept && !general_select(p);
            if (lane == 0 && !dr.zclear)
                st_u32(fl, 0u);
        } else {
            zb = ld_f32(&p.z[b]);
        }
    }
    if (general_select(p)) {
        // W > 1: the tiles' lists of length jsel, latest tile first: the first
        // W occurrences in that order are the W most recent
        const int W = p.W, T = p.scan_tiles;
        if (lane < W)
            sh.scan.merged[lane] = lane == 0 && mn > 0 ? me + 1 : 0;
        if (mn > 0 && W > 1) {
            const int32_t *cb = p.ws.cand + (int64_t)b * p.ws.cand_stride;
            int cnt = 0;
            for (int q0 = 0; q0 < T * W && cnt < W; q0 += 64) {
                const int q = q0 + lane;
                int v = 0;
                if (q < T * W) {
                    const int tq = q / W;
                    v = ld_i32(&cb[((T - 1 - tq) * SWITCHSD_MAX_NGRAM + jsel) * W + (q - tq * W)]);
                }
                const unsigned long long nz = __ballot(v > 0);
                const int rank = cnt + __popcll(nz & ((1ull << lane) - 1ull));
                if (v > 0 && rank < W)
                    sh.scan.merged[rank] = v;
                cnt += __popcll(nz);
            }
        }
        if (W > 1 && p.ws.cand_stride > 0) {
            // every tile's lists zeroed again: calls sharing a workspace carve
            // it by their own shapes, so a list left behind could sit under
            // another call's slots
            int32_t *cw = p.ws.cand + (int64_t)b * p.ws.cand_stride;
            for (int q = lane; q < T * SWITCHSD_MAX_NGRAM * W; q += 64)
                st_i32(&cw[q], 0);
        }
        const int v = lane < W ? sh.scan.merged[lane] : 0;
        front_finish_w(p, b, mn, v, L, zb, pre, sh, t0, t0 - 64 > 0 ? t0 - 64 : 0,
                       t0 + kScanTile < p.Lmax ? t0 + kScanTile : p.Lmax, dr);
        if (lane == 0 && !p.poll_front)
            st_u32(&p.ws.tk_front[b * kLineU32], 0u);
        return;
    }
    (void)in_tile;
    front_finish(p, b, mn, me, L, zb, pre, ct1, true, dr);
    if (lane == 0 && !p.poll_front)
        st_u32(&p.ws.tk_front[b * kLineU32], 0u);
}

// ------------------------------------------------------------- polling

__device__ __forceinline__ unsigned long long ld_slot(const unsigned long long *p) {
    return ld_u64(p);
}
__device__ __forceinline__ int32_t ld_slot(const int32_t *p) { return ld_i32(p); }

// Wave 0 polls workspace slots base[q * 64 + lane] (q < kQ) for the ones it
// waits for (bit q of want(), evaluated once the first round of requests is
// out, so that whatever it waits for overlaps with that round) until each
// holds a nonzero value, one round of requests at a time, each issued as soon
// as the previous one returned.  Every request is issued unconditionally
// (slots past n re-read slot n - 1): one load instruction per q and round,
// with no branch around it.  (Measured: keeping a second round in flight, or
// pausing between rounds, gains nothing and the former slows the step.)
// got[q] gets each slot's first nonzero value, 0 if `cap` rounds pass first
// (returns false then); rounds is the number of rounds after the first.
// on_miss() runs once, when the first round did not find every value.
template <typename T, int kQ, typename Want, typename Miss>
__device__ bool poll_slots(const T *base, int n, Want want, T (&got)[kQ], int cap, int &rounds,
                           Miss on_miss) {
    const int lane = threadIdx.x;
    T v[kQ];
    auto issue = [&]() {
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int i = q * 64 + lane;
            v[q] = ld_slot(base + (i < n ? i : n - 1));
        }
    };
    issue();
    uint32_t pend = want();
#pragma unroll
    for (int q = 0; q < kQ; ++q)
        got[q] = 0;
    for (int spin = 0;; ++spin) {
        rounds = spin;
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const bool hit = ((pend >> q) & 1u) != 0u && v[q] != 0;
            got[q] = hit ? v[q] : got[q];
            pend = hit ? pend & ~(1u << q) : pend;
        }
        if (__ballot(pend != 0u) == 0ull)
            return true;
        if (spin >= cap)
            return false;
        issue();
        if (spin == 0)
            on_miss();
    }
}

// poll_slots over n <= kMaxPollSlots slots with as few requests per lane as n
// allows; got[q] past them is 0.
template <typename T, typename Want, typename Miss>
__device__ bool poll_wave(const T *base, int n, Want want, T (&got)[8], int cap, int &rounds,
                          Miss on_miss) {
    if (n > 256)
        return poll_slots<T, 8>(base, n, want, got, cap, rounds, on_miss);
#pragma unroll
    for (int q = 0; q < 8; ++q)
        got[q] = 0;
    bool ok;
    if (n <= 64) {
        T g[1];
        ok = poll_slots<T, 1>(base, n, want, g, cap, rounds, on_miss);
        got[0] = g[0];
    } else {
        T g[4];
        ok = poll_slots<T, 4>(base, n, want, g, cap, rounds, on_miss);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            got[q] = g[q];
    }
    return ok;
}

// The last scan tile of sequence b when the tiles hand over through per-tile
// slots (poll_front): polls the other tiles' slots (tile t's length j at
// t * 8 + j, read by lane (t * 8 + j) mod 64, so lane j mod 8 always reads
// length j) until each holds its value, zeroes them again (at once, or with
// the front's outputs: DraftRegs), and folds them with this tile's own
// result; lane j < n_ngram gets the slot value of length j over all tiles.  The other tiles wait for nothing, so every slot is
// written in bounded time; the cap guards a broken launch, and on reaching it
// the sequence's error word is set and the missing tiles count as holding no
// occurrence.
__device__ int32_t poll_tiles(const StepParams &p, int b, const Shared &sh, DraftRegs &dr) {
    const int lane = threadIdx.x;
    const int n = (p.scan_tiles - 1) * SWITCHSD_MAX_NGRAM;  // <= kMaxPollSlots
    int32_t *ts = p.ws.tslot + (int64_t)b * p.ws.tslot_stride;
    const int j = lane & (SWITCHSD_MAX_NGRAM - 1);
    auto want = [&]() {  // bit q: slot q * 64 + lane is awaited
        uint32_t w = 0;
        for (int q = 0; q * 64 < n; ++q)
            if (q * 64 + lane < n && j < p.n_ngram)
                w |= 1u << q;
        return w;
    };
    int32_t got[8];
    int rounds = 0;
    if (!poll_wave(ts, n, want, got, p.spin_cap, rounds, [] {}) && lane == 0)
        st_u32(error_word(p, b), 1u);  // gave up: missing tiles hold no occurrence
    TL_ADD(6, (unsigned long long)(rounds + 1));
    int32_t best = 0;
    uint32_t seen = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q)
        if (got[q]) {
            best = got[q] - 1 > best ? got[q] - 1 : best;
            seen |= 1u << q;
        }
    // the slots are zeroed again now, or with the front's outputs after the
    // accept epilogue's poll (store_front)
    if (p.poll_accept && !general_select(p))
        dr.tclear = seen;
    else
        for (int q = 0; q < 8; ++q)
            if ((seen >> q) & 1u)
                st_i32(&ts[q * 64 + lane], 0);
#pragma unroll
    for (int o = SWITCHSD_MAX_NGRAM; o < 64; o <<= 1) {
        const int32_t y = __shfl_xor(best, o);
        best = y > best ? y : best;
    }
    if (lane < p.n_ngram) {
        const int32_t own = sh.scan.red[lane];
        return own > best ? own : best;
    }
    return 0;
}

__device__ __forceinline__ int32_t decode_key(unsigned long long key) {
    return key ? (int32_t)(0xFFFFFFFFu - (uint32_t)key) : 0;
}

// Accept and bonus of sequence b with R <= 64 nodes (Sec. 3.3, verification;
// tree drafts App. D), node i in lane i: its row maximum `key` (packed; 0
// none), its drafted token and parent, and the raw node count dn_raw.  Writes
// amax, out_tokens, accept_len, accept_node and bonus, and with kCommit the
// accepted tokens and the bonus into the context at cL; returns the accepted
// length (uniform over the wave).
template <bool kCommit>
__device__ int accept_lanes(const StepParams &p, int b, unsigned long long key, int tok, int par,
                            int dn_raw, int cL) {
    const int i = threadIdx.x;
    const int64_t base = (int64_t)b * p.R;
    const int64_t crow = (int64_t)b * p.Lmax;
    // output position j of the accepted path (then the bonus) holds v
    auto emit = [&](int j, int v) {
        p.out_tokens[base + j] = v;
        if (kCommit && cL + j < p.Lmax)
            p.ctok[crow + cL + j] = v;
    };
    const int dnb = clampi(dn_raw, 1, p.R);
    int a = -1;
    if (i < p.R) {
        if (i < dnb)
            a = decode_key(key);
        if (p.amax)
            p.amax[base + i] = a;
    }
    const bool valid = i >= 1 && i < dnb && par >= 0 && par < i;
    const int anc0 = valid ? par : 0;
    const int apar = __shfl(a, anc0);
    int ok = i == 0 ? 1 : (valid && tok == apar ? 1 : 0);
    int best, depth, dep;
    unsigned long long onpath;
    // a chain (every node's parent is the node before it): the accepted
    // nodes are the prefix before the first rejection
    const bool chain = __ballot(i >= 1 && i < dnb && par != i - 1) == 0ull;
    if (chain) {
        const unsigned long long rej = __ballot(i >= 1 && i < dnb && !ok);
        depth = rej ? __ffsll((long long)rej) - 2 : dnb - 1;
        best = depth;
        dep = i;
        onpath = depth > 0 ? (((~0ull) >> (64 - depth)) << 1) : 0ull;
    } else {
        dep = i == 0 ? 0 : 1;
        int anc = anc0;
#pragma unroll
        for (int round = 0; round < 6; ++round) {  // 2^6 >= 64 levels
            const int ok2 = __shfl(ok, anc), dep2 = __shfl(dep, anc),
                      anc2 = __shfl(anc, anc);
            ok &= ok2;
            dep += dep2;
            anc = anc2;
        }
        const uint32_t key2 =
            (ok && i < dnb) ? (((uint32_t)dep << 16) | (0xFFFFu - (uint32_t)i)) : 0u;
        const uint32_t kbest = wave_max_u32(key2);
        best = (int)(0xFFFFu - (kbest & 0xFFFFu));
        depth = (int)(kbest >> 16);
        onpath = 0ull;
        int cur = best;
        for (int s2 = 0; s2 < depth; ++s2) {
            onpath |= 1ull << cur;
            cur = __shfl(anc0, cur);
        }
    }
    const int bon = __shfl(a, best);
    if (i < p.R) {
        if ((onpath >> i) & 1ull)
            emit(dep - 1, tok);
        if (i == depth)
            emit(i, bon);
        else if (i > depth)
            p.out_tokens[base + i] = -1;
    }
    if (i == 0) {
        p.accept_len[b] = depth;
        p.accept_node[b] = best;
        p.bonus[b] = bon;
    }
    return depth;
}

// Decode loop: the context's new length and the draft model's position after
// a step that accepted acc tokens (lane 0).
__device__ __forceinline__ void commit_lengths(const StepParams &p, int b, int cL, int cdp,
                                               int cuc, int acc) {
    const int Lnew = cL + acc + 1 < p.Lmax ? cL + acc + 1 : p.Lmax;
    const int pos = clampi(cuc ? cdp : cL + acc, 0, Lnew);
    p.clen[b] = Lnew;
    p.draft_pos[b] = pos;
    p.lag[b] = Lnew - pos;
}

// kCommit: the decode loop's commit is compiled in.
template <bool kCommit>
__device__ void final_epilogue(const StepParams &p, int b, Shared &sh) {
    const int lane = threadIdx.x;
    const int64_t base = (int64_t)b * p.R;
    unsigned long long *keys = p.ws.keys + (int64_t)b * p.ws.key_stride;
    // decode loop (Sec. 3.3, KV Cache Synchronization): the accepted tokens and
    // the bonus also go to the context at its length cL
    int cL = 0, cdp = 0, cuc = 0;
    if (kCommit) {
        cL = clampi(p.clen[b], 0, p.Lmax);
        cdp = p.draft_pos[b];
        cuc = ld_i32(&p.use_copy[b]);
    }
    const int64_t crow = (int64_t)b * p.Lmax;
    // output position j of the accepted path (then the bonus) holds v
    auto emit = [&](int j, int v) {
        p.out_tokens[base + j] = v;
        if (kCommit && cL + j < p.Lmax)
            p.ctok[crow + cL + j] = v;
    };
    int acc = 0;  // accepted length (uniform over the wave)
    if (p.R <= 64) {
        const int i = lane;
        // the draft and the row maxima, all requested at once
        const int dn_raw = ld_i32(&p.dn[b]);
        unsigned long long key = 0ull;
        int tok = -1, par = -1;
        if (i < p.R) {
            key = ld_u64(&keys[i]);
            tok = ld_i32(&p.dtok[base + i]);
            par = p.dpar ? ld_i32(&p.dpar[base + i]) : i - 1;
        }
#ifdef SWITCHSD_TIMELINE
        __builtin_amdgcn_s_waitcnt(0);
#endif
        TL_MARK(5);
        if (i < p.R && key)
            st_u64(&keys[i], 0ull);
        acc = accept_lanes<kCommit>(p, b, key, tok, par, dn_raw, cL);
    } else {
        const int dnb = clampi(ld_i32(&p.dn[b]), 1, p.R);
        // the draft and the row maxima into LDS, 256 nodes at a time with all
        // of their loads in flight together
        for (int i0 = 0; i0 < p.R; i0 += 4 * 64) {
            unsigned long long kq[4];
            int tq[4], pq[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = i0 + lane + 64 * q;
                kq[q] = 0ull;
                tq[q] = -1;
                pq[q] = -1;
                if (i < p.R) {
                    kq[q] = ld_u64(&keys[i]);
                    tq[q] = ld_i32(&p.dtok[base + i]);
                    pq[q] = p.dpar ? ld_i32(&p.dpar[base + i]) : i - 1;
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = i0 + lane + 64 * q;
                if (i < p.R) {
                    if (kq[q])
                        st_u64(&keys[i], 0ull);
                    const int a = i < dnb ? decode_key(kq[q]) : -1;
                    sh.epi.a[i] = a;
                    sh.epi.tok[i] = tq[q];
                    sh.epi.par[i] = pq[q];
                    if (p.amax)
                        p.amax[base + i] = a;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        // key of the deepest accepted node, ties to the lowest index:
        // (depth << 16) | (0xFFFF - node); the anchor's is 0xFFFF
        uint32_t kb = lane == 0 ? 0xFFFFu : 0u;
        bool other = false;  // some node hangs off neither the anchor nor its predecessor
        for (int i = lane; i < dnb; i += 64) {
            const int q = sh.epi.par[i];
            other |= i >= 1 && q != 0 && q != i - 1;
        }
        if (__ballot(other) == 0ull) {
            // Runs of consecutive nodes, each starting at a child of the
            // anchor (one chain, or W copy candidates): node i is accepted iff
            // no edge fails between the start of its run and i, and its depth
            // is its distance to that start.  One ballot pair per 64 nodes.
            int S = 0, F = -1;  // last run start / failed edge of earlier blocks
            for (int i0 = 0; i0 < dnb; i0 += 64) {
                const int i = i0 + lane;
                bool st = false, fl = false;
                if (i >= 1 && i < dnb) {
                    const int q = sh.epi.par[i];
                    st = q == 0;
                    fl = sh.epi.tok[i] != sh.epi.a[q];
                }
                const unsigned long long sm = __ballot(st), fm = __ballot(fl);
                const unsigned long long le = lane == 63 ? ~0ull : ((2ull << lane) - 1ull);
                const int si = (sm & le) ? i0 + 63 - __clzll((long long)(sm & le)) : S;
                const int fi = (fm & le) ? i0 + 63 - __clzll((long long)(fm & le)) : F;
                if (i >= 1 && i < dnb && fi < si) {
                    const uint32_t key2 =
                        ((uint32_t)(i - si + 1) << 16) | (0xFFFFu - (uint32_t)i);
                    kb = key2 > kb ? key2 : kb;
                }
                if (sm)
                    S = i0 + 63 - __clzll((long long)sm);
                if (fm)
                    F = i0 + 63 - __clzll((long long)fm);
            }
        } else {
            // Pointer jumping over the nodes below dnb.  State of node i: bit 31
            // = every edge from i up to `anc` holds, bits 16..30 = the number of
            // those edges, bits 0..15 = anc.  Initially anc is the parent (the
            // anchor for node 0 and for a node without a valid parent, which also
            // fails its edge); each round replaces the state by its composition
            // with the state of anc, doubling the covered path, until every path
            // reaches the anchor, whose state (holds, 0 edges, itself) is the
            // identity.
            bool open = false;  // some path of this lane's nodes not yet at the anchor
            for (int i = lane; i < dnb; i += 64) {
                const int q = sh.epi.par[i];
                const bool valid = i >= 1 && q >= 0 && q < i;
                const bool ok = i == 0 || (valid && sh.epi.tok[i] == sh.epi.a[q]);
                sh.epi.st[0][i] = (ok ? 0x80000000u : 0u) | ((i == 0 ? 0u : 1u) << 16) |
                                  (uint32_t)(valid ? q : 0);
                open |= valid && q != 0;
            }
            __builtin_amdgcn_wave_barrier();
            int cur = 0;
            while (__ballot(open)) {
                const uint32_t *from = sh.epi.st[cur];
                uint32_t *to = sh.epi.st[cur ^ 1];
                open = false;
                for (int i0 = 0; i0 < dnb; i0 += 4 * 64) {
                    uint32_t s1[4], s2[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int i = i0 + lane + 64 * q;
                        s1[q] = i < dnb ? from[i] : 0u;
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        s2[q] = from[s1[q] & 0xFFFFu];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int i = i0 + lane + 64 * q;
                        if (i < dnb) {
                            const uint32_t nv =
                                (s1[q] & s2[q] & 0x80000000u) |
                                ((s1[q] & 0x7FFF0000u) + (s2[q] & 0x7FFF0000u)) |
                                (s2[q] & 0xFFFFu);
                            to[i] = nv;
                            open |= (nv & 0xFFFFu) != 0u;
                        }
                    }
                }
                cur ^= 1;
                __builtin_amdgcn_wave_barrier();
            }
            // deepest accepted node
            for (int i = lane; i < dnb; i += 64) {
                const uint32_t s1 = sh.epi.st[cur][i];
                if (s1 >> 31) {
                    const uint32_t key2 =
                        (((s1 >> 16) & 0x7FFFu) << 16) | (0xFFFFu - (uint32_t)i);
                    kb = key2 > kb ? key2 : kb;
                }
            }
        }
        kb = wave_max_u32(kb);
        const int best = (int)(0xFFFFu - (kb & 0xFFFFu));
        const int depth = (int)(kb >> 16);
        const int bon = sh.epi.a[best];
        for (int i = lane; i < p.R; i += 64)
            if (i > depth)
                p.out_tokens[base + i] = -1;
        // the path is usually one run of consecutive nodes (a chain, or one
        // copy candidate): then write it in parallel, else walk it
        const int first = best - depth + 1;
        bool bad = false;
        for (int j = lane; j < depth; j += 64) {
            const int node = first + j;
            bad |= node < 1 || sh.epi.par[node] != (j == 0 ? 0 : node - 1);
        }
        if (__ballot(bad) == 0ull) {
            for (int j = lane; j < depth; j += 64)
                emit(j, sh.epi.tok[first + j]);
        } else if (lane == 0) {
            int cur = best;
            for (int pos = depth - 1; pos >= 0; --pos) {
                emit(pos, sh.epi.tok[cur]);
                cur = sh.epi.par[cur];
            }
        }
        if (lane == 0) {
            emit(depth, bon);
            p.accept_len[b] = depth;
            p.accept_node[b] = best;
            p.bonus[b] = bon;
        }
        acc = depth;
    }
    if (kCommit && lane == 0)
        commit_lengths(p, b, cL, cdp, cuc, acc);
    if (lane == 0)
        st_u32(&p.ws.tk_all[b * kLineU32], 0u);
}

// Row maxima of sequence b in the fused step with per-segment slots (wave 0
// of the work-group that chose the draft; R <= 64, R * segs <= kMaxPollSlots):
// lane r gets the maximum over the segments of row r (0: no candidate, or a
// row that is not verified).  Slot j = s * R + r is read by lane j mod 64;
// every slot of a needed row is polled until it holds its segment's result
// (nonzero), then zeroed again.  The argmax work-groups wait for nothing, so the results
// arrive in bounded time; the cap guards a broken launch, and on reaching it
// the sequence's error word is set and the missing results count as none.
template <typename Miss>
__device__ unsigned long long poll_rows(const StepParams &p, int b, int nnb, Shared &sh,
                                        Miss on_miss) {
    const int lane = threadIdx.x;
    const int R = p.R, n = R * p.segs;  // <= kMaxPollSlots
    unsigned long long *sk = p.ws.skeys + (int64_t)b * p.ws.skey_stride;
    unsigned long long *lk = sh.poll.k;
    TL_MARK(5);
    int need = 0;
    uint32_t want = 0;
    auto wantf = [&]() {  // bit q: slot q * 64 + lane is awaited
        need = (int)rows_of_drafts(p, nnb);  // as rows_needed, nn[b] already read
        want = 0;
        for (int q = 0, r = lane % R; q * 64 < n; ++q, r = (r + 64) % R)
            if (q * 64 + lane < n && r < need)
                want |= 1u << q;
        return want;
    };
    unsigned long long got[8];
    int rounds = 0;
    if (!poll_wave(sk, n, wantf, got, p.spin_cap, rounds, on_miss) && lane == 0)
        st_u32(error_word(p, b), 1u);  // gave up: missing segments hold no maximum
    TL_ADD(6, (unsigned long long)(rounds + 1) << 32);
#pragma unroll
    for (int q = 0; q < 8; ++q)
        if ((want >> q) & 1u) {
            lk[q * 64 + lane] = got[q];
            if (got[q])
                st_u64(&sk[q * 64 + lane], 0ull);
        }
    __builtin_amdgcn_wave_barrier();
    unsigned long long key = 0ull;
    if (lane < need)
        for (int sg = 0; sg < p.segs; ++sg) {
            const unsigned long long v = lk[sg * R + lane];
            key = v > key ? v : key;
        }
    return key > 1ull ? key : 0ull;
}

// The fused step's accept epilogue from the work-group that chose the draft
// (still in registers, dr): polls the segment results, then accept, bonus and
// the decode loop's commit as in final_epilogue.
template <bool kCommit>
__device__ void poll_epilogue(const StepParams &p, int b, const DraftRegs &dr, Shared &sh) {
    int cL = 0, cdp = 0;
    if (kCommit) {
        cL = clampi(p.clen[b], 0, p.Lmax);
        cdp = p.draft_pos[b];
    }
    // the front's deferred outputs go out once the first poll round has
    // returned without every result (they then complete while the poll goes
    // on), else with the accept's outputs
    bool stored = !dr.deferred;
    const unsigned long long key = poll_rows(p, b, dr.nnb, sh, [&] {
        if (!stored) {
            store_front(p, b, dr, true);
            stored = true;
        }
    });
    TL_MARK(3);
    if (!stored)
        store_front(p, b, dr, true);
    const int acc = accept_lanes<kCommit>(p, b, key, dr.tok, dr.par, dr.dn, cL);
    if (kCommit && threadIdx.x == 0)
        commit_lengths(p, b, cL, cdp, dr.use, acc);
}

// The verify launch's waiting work-group of sequence b (wave 0; R <= 64):
// the draft, written by an earlier launch, read into registers while the
// argmax work-groups stream (its accept epilogue then polls their results).
template <bool kCommit>
__device__ __forceinline__ void poller_draft(const StepParams &p, int b, DraftRegs &dr) {
    const int lane = threadIdx.x;
    const int64_t base = (int64_t)b * p.R;
    const int dn_raw = p.dn[b];
    if (lane < p.R) {
        dr.tok = p.dtok[base + lane];
        dr.par = p.dpar ? p.dpar[base + lane] : lane - 1;
    }
    dr.dn = dn_raw;
    dr.nnb = clampi(dn_raw, 1, p.R);  // the rows the argmax work-groups verify
    if (kCommit)
        dr.use = p.use_copy[b];
}

// ------------------------------------------------------------- streamed verify

// Arrival of n units of work at a ticket expecting `expected` in all (wave 0).
__device__ __forceinline__ bool arrive_n(uint32_t *ticket, uint32_t n, uint32_t expected) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0);
    uint32_t old = 0;
    if (threadIdx.x == 0)
        old = __hip_atomic_fetch_add(ticket, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    old = __shfl(old, 0);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    return old + n == expected;
}

// Verify over the drafted rows only, for 16-byte aligned rows (V % 8 == 0 and
// an aligned tensor).  The units of work are the 16 KB chunks of the rows
// r < dn[b], sequence by sequence, row by row (p.segs chunks per row); work-
// group g streams the contiguous units [U g / G, U (g + 1) / G) with the next
// chunk in flight while one is reduced, across row boundaries.  At the end of
// a row piece each wave max-combines its (value, index) into the row's key; at
// the end of a sequence piece the work-group arrives with its unit count, and
// the last arrival (dn[b] * chunks per row in all) runs the accept epilogue.
template <bool kCommit>
__device__ void verify_stream(const StepParams &p, Shared &sh, u32x4 *keep) {
    const int tid = threadIdx.x, lane = tid & 63;
    constexpr int Q = kListMaxB / 64;
    const int cpr = p.segs;
    // first unit of sequence b = lane + 64 q (exclusive prefix) and its dn
    int first[Q], dnq[Q];
    int carry = 0;
    // (every load issued before any is used: the addresses are clamped rather
    // than the loads made conditional, which would wait for each in turn)
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int b = lane + 64 * q;
        dnq[q] = ld_i32(&p.dn[b < p.B ? b : p.B - 1]);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q)
        dnq[q] = lane + 64 * q < p.B ? clampi(dnq[q], 1, p.R) : 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int cnt = dnq[q] * cpr;
        int inc = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(inc, o);
            if (lane >= o)
                inc += y;
        }
        first[q] = carry + inc - cnt;
        carry += __shfl(inc, 63);
    }
    const int64_t U = carry;
    const int u0 = (int)(U * blockIdx.x / gridDim.x), u1 = (int)(U * (blockIdx.x + 1) / gridDim.x);
    if (u0 >= u1)
        return;
    // coordinates of unit u0: the last sequence starting at or before it
    int b = 0, fb = 0, dnb = 1;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const unsigned long long m = __ballot(lane + 64 * q < p.B && first[q] <= u0);
        if (m) {
            const int l = 63 - __clzll((long long)m);
            b = 64 * q + l;
            fb = __shfl(first[q], l);
            dnb = __shfl(dnq[q], l);
        }
    }
    int r = (u0 - fb) / cpr, c = u0 - fb - r * cpr;
    const int nq = p.V >> 3;
    auto row_vecs = [&](int bb, int rr) {
        return reinterpret_cast<const u32x4 *>(p.logits + ((int64_t)bb * p.R + rr) * p.V);
    };
    u32x4 A[kUnroll], Bv[kUnroll];
    load_chunk(A, row_vecs(b, r), c * kChunkVecs, nq);
    LazyMaxLds st;
    st.d = keep;
    lazy_init(st);
    for (int u = u0; u < u1; ++u) {
        // the next unit
        int nb = b, nr = r, nc = c + 1, ndn = dnb;
        if (nc == cpr) {
            nc = 0;
            if (++nr == dnb) {
                nr = 0;
                ++nb;
                if (u + 1 < u1) {  // the next sequence's dn (identical in every lane)
                    const int q = nb >> 6, l = nb & 63;
                    int v = 0;
#pragma unroll
                    for (int qq = 0; qq < Q; ++qq)
                        if (qq == q)
                            v = __shfl(dnq[qq], l);
                    ndn = v;
                }
            }
        }
        if (u + 1 < u1)
            load_chunk(Bv, row_vecs(nb, nr), nc * kChunkVecs, nq);
        lazy_chunk(A, c * kChunkVecs, nq, st);
        const bool last_unit = u + 1 == u1;
        if (c == cpr - 1 || last_unit) {  // end of this row's piece
            float runM;
            const uint32_t runI = wave_argmax(st.best, lazy_index(st, nq, 0u), runM);
            if (lane == 0 && runI != kNoIdx) {
                const unsigned long long key =
                    ((unsigned long long)order_key(runM) << 32) | (0xFFFFFFFFu - runI);
                atomicMax(&p.ws.keys[(int64_t)b * p.ws.key_stride + r], key);
            }
            lazy_init(st);
        }
        b = nb;
        r = nr;
        c = nc;
        dnb = ndn;
#pragma unroll
        for (int q = 0; q < kUnroll; ++q)
            A[q] = Bv[q];
    }
    if (!p.epi_accept)
        return;
    // The arrivals, once the whole stream is done: one per sequence this
    // work-group streamed a piece of, lane b mod 64 arriving for sequence b
    // with the piece's unit count, all in one round trip.  (Arriving at each
    // sequence's end inside the stream waited there for the chunk in flight
    // and the atomic's round trip.)  The sequences whose last arrival this
    // was then run their accept epilogues.
    __builtin_amdgcn_s_waitcnt(0);  // this wave's row-key atomics are done
    __syncthreads();
    if (tid >= 64)
        return;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    unsigned long long pend[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int bq = lane + 64 * q;
        const int e = first[q] + dnq[q] * cpr;
        const int n = (u1 < e ? u1 : e) - (u0 > first[q] ? u0 : first[q]);
        bool last = false;
        if (bq < p.B && n > 0) {
            const uint32_t old = __hip_atomic_fetch_add(&p.ws.tk_all[bq * kLineU32], (uint32_t)n,
                                                        __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            last = old + (uint32_t)n == (uint32_t)(dnq[q] * cpr);
        }
        pend[q] = __ballot(last);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
    for (int q = 0; q < Q; ++q)
        for (unsigned long long m = pend[q]; m != 0ull; m &= m - 1ull)
            final_epilogue<kCommit>(p, 64 * q + __ffsll((long long)m) - 1, sh);
}

// ------------------------------------------------------------- draws at T > 0

// Sampling temperature T > 0 (App. A).  The target's distribution at a
// drafted row is p = softmax(l / T), realized with integer weights
// w_j = floor(2^40 * 2^((l_j - m) c)), c = log2(e) / T, m the row maximum, so
// that every sum is exact and the drawn index does not depend on the order
// of the reduction.  One-hot drafts (copy drafts, trees, drafts without their
// distribution): speculative sampling emits the same token law as drawing y
// from p at each drafted row and accepting a child iff its token is y.  Two
// launches after the draft is chosen: the row maxima (the greedy argmax
// pass), then the per-chunk weight sums, whose last work-group per row draws
// the row's token and whose last row closes the sequence with the accept
// epilogue.

// The row's maximum from its packed argmax key; false when the row has no
// finite maximum (no key: every value NaN; -inf; +inf present), and then the
// row keeps the greedy choice (its weights are one-hot there).
__device__ __forceinline__ bool key_max(unsigned long long key, float &m) {
    if (!key)
        return false;
    const uint32_t k = (uint32_t)(key >> 32);
    m = __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
    return __builtin_isfinite(m);
}

// floor(2^40 * 2^t) for t = (l - m) c as a float (an integer <= 2^40): 2^t =
// 2^k * P(t - k), k = rint(t), P the degree-6 Taylor polynomial of 2^f =
// e^(f ln 2) on [-1/2, 1/2] by Horner's rule in fused multiply-adds.  The
// coefficients carry the factor 2^40 (a power-of-two scaling commutes with
// every rounding here), and t is clamped to >= -41 (every t below, NaN
// included, then gives 2^40 * 2^-41 = 1/2, which floors to 0, as the weight
// of any t < -40.5 does).
__device__ __forceinline__ float samp_weight(float l, float m, float c) {
    const float t = __builtin_fmaxf((l - m) * c, -41.0f);
    const float k = __builtin_rintf(t);
    const float f = t - k;
    float q = 0x1.430912p+27f;                  // 2^40 ln2^6 / 6!
    q = __builtin_fmaf(q, f, 0x1.5d87fep+30f);  // 2^40 ln2^5 / 5!
    q = __builtin_fmaf(q, f, 0x1.3b2ab6p+33f);  // 2^40 ln2^4 / 4!
    q = __builtin_fmaf(q, f, 0x1.c6b08ep+35f);  // 2^40 ln2^3 / 3!
    q = __builtin_fmaf(q, f, 0x1.ebfbe0p+37f);  // 2^40 ln2^2 / 2!
    q = __builtin_fmaf(q, f, 0x1.62e430p+39f);  // 2^40 ln2
    q = __builtin_fmaf(q, f, 0x1p+40f);         // 2^40
    return __builtin_floorf(__builtin_ldexpf(q, (int)k));
}

// Weight sum of the 8 elements of one 16-byte vector (< 2^44, exact: every
// partial sum is an integer below 2^53).
__device__ __forceinline__ double vec_weight(const u32x4 &v, float m, float c) {
    double s = 0.0;
#pragma unroll
    for (int w4 = 0; w4 < 4; ++w4)
        s += (double)samp_weight(lo_f(v[w4]), m, c) + (double)samp_weight(hi_f(v[w4]), m, c);
    return s;
}

// Wave sum of doubles holding integers below 2^53 (every partial sum exact,
// so the result does not depend on the reduction order): DPP row shifts and
// row broadcasts on both halves, as wave_reduce_u32.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_shift_f64(double v) {
    const unsigned long long u = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, kCtrl, kRowMask, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), kCtrl, kRowMask, 0xf,
                                               false);
    return __longlong_as_double((long long)(((unsigned long long)(uint32_t)hi << 32) |
                                            (uint32_t)lo));
}
__device__ __forceinline__ double wave_sum_f64(double v) {
    v += dpp_shift_f64<0x111, 0xf>(v);
    v += dpp_shift_f64<0x112, 0xf>(v);
    v += dpp_shift_f64<0x114, 0xf>(v);
    v += dpp_shift_f64<0x118, 0xf>(v);
    v += dpp_shift_f64<0x142, 0xa>(v);
    v += dpp_shift_f64<0x143, 0xc>(v);
    const unsigned long long u = __double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Inclusive prefix sum of 64-bit integers over the 64 lanes of a wave, in DPP
// moves (no LDS): row shifts by 1, 2, 4 and 8 within each row of 16 lanes,
// then lane 15's total into rows 1 and 3 and lane 31's into rows 2 and 3 (as
// wave_sum_f64, whose lane 63 is the total).  kSteps < 6 stops after the
// first kSteps (e.g. 3: the prefix of lanes 0..7 of row 0).
template <int kCtrl, int kRowMask>
__device__ __forceinline__ unsigned long long dpp_shift_u64(unsigned long long v) {
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, kCtrl, kRowMask, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), kCtrl, kRowMask, 0xf,
                                               false);
    return ((unsigned long long)(uint32_t)hi << 32) | (uint32_t)lo;
}
template <int kSteps = 6>
__device__ __forceinline__ unsigned long long wave_scan_u64(unsigned long long v) {
    v += dpp_shift_u64<0x111, 0xf>(v);
    v += dpp_shift_u64<0x112, 0xf>(v);
    v += dpp_shift_u64<0x114, 0xf>(v);
    if (kSteps > 3)
        v += dpp_shift_u64<0x118, 0xf>(v);
    if (kSteps > 4)
        v += dpp_shift_u64<0x142, 0xa>(v);
    if (kSteps > 5)
        v += dpp_shift_u64<0x143, 0xc>(v);
    return v;
}
// Lane l's value (l uniform over the wave).
__device__ __forceinline__ unsigned long long readlane_u64(unsigned long long v, int l) {
    l = __builtin_amdgcn_readfirstlane(l);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((unsigned long long)hi << 32) | lo;
}

// floor(u * Z / 2^64), exactly (the upper half of the 128-bit product).
__device__ __forceinline__ unsigned long long scaled_target(unsigned long long u,
                                                            unsigned long long Z) {
    return __umul64hi(u, Z);
}

// The sum launch reads each chunk wave by wave: the kUnroll * 64 vectors of
// wave w in chunk c are contiguous, [c kChunkVecs + 256 w, + 256), vector u of
// lane l at 64 u + l; one weight sum per (chunk, wave) then covers a
// contiguous range in index order.
__device__ __forceinline__ void load_chunk_w(u32x4 (&v)[kUnroll], const u32x4 *vp, int qc0,
                                             int nq) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int q = qc0 + wave * (kUnroll * 64) + u * 64 + lane;
        v[u] = __builtin_nontemporal_load(vp + (q < nq ? q : nq - 1));
    }
}

// Weight sums of chunk c (16 KB) of a row, one per wave (its contiguous 256
// vectors), stored at cs[c * kWaves + wave] (plus `mark`: 1 where a poller
// tells a written sum from an empty slot); the entries of a row in index
// order are chunk by chunk, wave by wave.
__device__ __forceinline__ void store_block_sums(const u32x4 (&A)[kUnroll], int c, int nq, float m,
                                                 float samp_c, unsigned long long *cs,
                                                 unsigned long long mark) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int q0 = c * kChunkVecs + wave * (kUnroll * 64) + lane;
    double w = 0.0;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        w += q0 + u * 64 < nq ? vec_weight(A[u], m, samp_c) : 0.0;
    w = wave_sum_f64(w);
    if (lane == 0)
        __hip_atomic_store(&cs[c * kWaves + wave], (unsigned long long)w + mark,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The draw of row r of sequence b (its maximum m), by wave 0: the (chunk,
// wave) sums give Z and the target floor(u Z / 2^64), then the chunk and the
// wave's 256 vectors holding it; only those are read again (four per lane),
// and the block of 64 vectors, the vector and the element are found by
// prefix sums over their weights.  The drawn token replaces the row's key
// (key_max reads it as a finite maximum of index y).  Every thread of the
// work-group calls this (the sums are staged in LDS by all of them).
__device__ void pick_row(const StepParams &p, int b, int r, float m, unsigned long long *keyp,
                         Shared &sh) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const unsigned long long *cs = p.csum + ((int64_t)b * p.R + r) * p.cpr * kWaves;
    const int ncs = p.cpr * kWaves;  // <= 256 (V <= 524288)
    for (int i = tid; i < ncs; i += kThreads)
        sh.pick.cw[i] = __hip_atomic_load(&cs[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (wave != 0)
        return;
    const unsigned long long uni = p.uniforms[(int64_t)b * p.R + r];
    // chunk totals, their inclusive prefix, the target and its chunk
    unsigned long long cc = 0;
    if (lane < p.cpr) {
#pragma unroll
        for (int e = 0; e < kWaves; ++e)
            cc += sh.pick.cw[lane * kWaves + e];
    }
    const unsigned long long inc = wave_scan_u64(cc);
    const unsigned long long Z = __shfl(inc, 63);
    unsigned long long tg = scaled_target(uni, Z);
    const unsigned long long hit = __ballot(lane < p.cpr && inc > tg);
    const int cst = __ffsll((long long)hit) - 1;  // exists: target < Z
    tg -= __shfl(inc - cc, cst);
    // the wave entry of that chunk holding the target (lanes 0..kWaves-1)
    const unsigned long long ce = lane < kWaves ? sh.pick.cw[cst * kWaves + lane] : 0ull;
    const unsigned long long ie = wave_scan_u64<3>(ce);
    const unsigned long long hit2 = __ballot(lane < kWaves && ie > tg);
    const int est = __ffsll((long long)hit2) - 1;  // exists: tg < the chunk's total
    tg -= __shfl(ie - ce, est);
    // the entry's 256 vectors, block u of 64 at 64 u + lane
    const int nq = p.V >> 3;
    const int q0 = cst * kChunkVecs + est * (kUnroll * 64) + lane;
    const u32x4 *vp = reinterpret_cast<const u32x4 *>(p.logits + ((int64_t)b * p.R + r) * p.V);
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        v[u] = q0 + u * 64 < nq ? vp[q0 + u * 64] : u32x4{0u, 0u, 0u, 0u};
    unsigned long long vw[kUnroll], bs[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        vw[u] = q0 + u * 64 < nq ? (unsigned long long)vec_weight(v[u], m, p.samp_c) : 0ull;
        bs[u] = (unsigned long long)wave_sum_f64((double)vw[u]);
    }
    // the block holding the target (exists: tg < the entry's total)
    int us = kUnroll - 1;
    unsigned long long incl = 0, us_before = 0;
    bool found = false;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const unsigned long long excl = incl;
        incl += bs[u];
        if (!found && tg < incl) {
            found = true;
            us = u;
            us_before = excl;
        }
    }
    tg -= us_before;
    unsigned long long w = 0;
    u32x4 x = v[0];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (u == us) {
            w = vw[u];
            x = v[u];
        }
    const unsigned long long iv = wave_scan_u64(w);
    const unsigned long long hit3 = __ballot(iv > tg);
    const int lst = __ffsll((long long)hit3) - 1;  // exists: tg < the block's total
    if (lane == lst) {
        // the element within this lane's vector
        unsigned long long run = iv - w;
        int e = 7;
        for (int j = 0; j < 8; ++j) {
            const uint32_t xj = x[j >> 1];
            run += (unsigned long long)samp_weight((j & 1) ? hi_f(xj) : lo_f(xj), m, p.samp_c);
            if (run > tg) {
                e = j;
                break;
            }
        }
        const uint32_t y = (uint32_t)(q0 + us * 64) * 8u + (uint32_t)e;
        st_u64(keyp, (1ull << 32) | (unsigned long long)(0xFFFFFFFFu - y));
    }
}

// ------------------------------------------------------------- speculative sampling with q

typedef unsigned __int128 u128;

// The wave's total of 64-bit integers (every lane).
__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
    return readlane_u64(wave_scan_u64(v), 63);
}
// Lane l's 128-bit value (l uniform over the wave).
__device__ __forceinline__ u128 readlane_u128(u128 v, int l) {
    return ((u128)readlane_u64((unsigned long long)(v >> 64), l) << 64) |
           readlane_u64((unsigned long long)v, l);
}
// Inclusive prefix sum of 128-bit integers over the lanes, in DPP moves as
// wave_scan_u64 (kSteps < 6: the first kSteps shifts only).
template <int kCtrl, int kRowMask>
__device__ __forceinline__ u128 dpp_shift_u128(u128 v) {
    return ((u128)dpp_shift_u64<kCtrl, kRowMask>((unsigned long long)(v >> 64)) << 64) |
           dpp_shift_u64<kCtrl, kRowMask>((unsigned long long)v);
}
template <int kSteps = 6>
__device__ __forceinline__ u128 wave_scan_u128(u128 v) {
    v += dpp_shift_u128<0x111, 0xf>(v);
    v += dpp_shift_u128<0x112, 0xf>(v);
    v += dpp_shift_u128<0x114, 0xf>(v);
    if (kSteps > 3)
        v += dpp_shift_u128<0x118, 0xf>(v);
    if (kSteps > 4)
        v += dpp_shift_u128<0x142, 0xa>(v);
    if (kSteps > 5)
        v += dpp_shift_u128<0x143, 0xc>(v);
    return v;
}
// The wave's total of 128-bit integers (every lane).
__device__ __forceinline__ u128 wave_sum_u128(u128 v) {
    return readlane_u128(wave_scan_u128(v), 63);
}
// Upper 128 bits of the 192-bit product a * b.
__device__ __forceinline__ u128 mulhi_128_64(u128 a, unsigned long long b) {
    const u128 lo = (u128)(unsigned long long)a * b;
    const u128 hi = (u128)(unsigned long long)(a >> 64) * b;
    return hi + (lo >> 64);
}

// One row's two distributions: the target's p (row maxima in keys, weight
// sums in csum) and the draft's q (qkeys, qcsum).  A row without a finite
// maximum has one-hot weights 2^40 at its greedy choice g.
struct SpecRow {
    float mp, mq;
    bool ap, aq;
    int gp, gq;
    unsigned long long Zp, Zq;
};

// Every lane of a wave ends with the row's SpecRow.
__device__ void spec_row_setup(const StepParams &p, int b, int r, SpecRow &s) {
    const int lane = threadIdx.x & 63;
    const unsigned long long kp = ld_u64(&p.ws.keys[(int64_t)b * p.ws.key_stride + r]);
    const unsigned long long kq = ld_u64(&p.ws.qkeys[(int64_t)b * p.ws.key_stride + r]);
    s.mp = s.mq = 0.0f;
    s.ap = key_max(kp, s.mp);
    s.aq = key_max(kq, s.mq);
    s.gp = decode_key(kp);
    s.gq = decode_key(kq);
    const int ncs = p.cpr * kWaves;
    const int64_t off = ((int64_t)b * p.R + r) * ncs;
    unsigned long long zp = 0, zq = 0;
    for (int i = lane; i < ncs; i += 64) {
        zp += __hip_atomic_load(&p.csum[off + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        zq += __hip_atomic_load(&p.qcsum[off + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    zp = wave_sum_u64(zp);
    zq = wave_sum_u64(zq);
    s.Zp = s.ap ? zp : 1ull << 40;
    s.Zq = s.aq ? zq : 1ull << 40;
}

// Integer weight of element j (value bits h) of a row with maximum m, or of a
// row without a finite maximum (one-hot 2^40 at g).
__device__ __forceinline__ unsigned long long elem_weight(float l, bool act, float m, int j, int g,
                                                          float c) {
    return act ? (unsigned long long)samp_weight(l, m, c) : (j == g ? 1ull << 40 : 0ull);
}

// The speculative-sampling test at row r of sequence b (wave 0): the drafted
// token x = dtok[b, r + 1] is accepted with probability min(1, p(x) / q(x)),
// i.e. iff u Q_x Zp < 2^64 P_x Zq in exact integers (u the row's accept
// uniform; a token outside [0, V) has P_x = Q_x = 0 and is rejected).
__device__ void spec_test(const StepParams &p, int b, int r) {
    SpecRow sr;
    spec_row_setup(p, b, r, sr);
    const int64_t row = (int64_t)b * p.R + r;
    const int x = ld_i32(&p.dtok[row + 1]);
    unsigned long long Px = 0, Qx = 0;
    if (x >= 0 && x < p.V) {
        Px = elem_weight(lo_f((uint32_t)p.logits[row * p.V + x]), sr.ap, sr.mp, x, sr.gp,
                         p.samp_c);
        Qx = elem_weight(lo_f((uint32_t)p.qlogits[row * p.V + x]), sr.aq, sr.mq, x, sr.gq,
                         p.samp_c);
    }
    const unsigned long long u = p.accept_uniforms[row];
    // u Q_x Zp = (hi, lo) with hi its upper 128 bits; 2^64 P_x Zq = (P_x Zq, 0)
    const u128 lhs_hi = mulhi_128_64((u128)u * Qx, sr.Zp);
    const bool acc = lhs_hi < (u128)Px * sr.Zq;
    if ((threadIdx.x & 63) == 0) {
        // the row's sums, for the residual launch should this row end the chain
        __hip_atomic_store(&p.rz[2 * row], sr.Zp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&p.rz[2 * row + 1], sr.Zq, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        st_u32(&p.rdec[row], acc ? 1u : 2u);
    }
}

// The sum work-groups of a drafted row arrive with the units (16 KB chunks or
// work-groups) they covered.  The last one either takes the row's accept test
// (a row with a drafted child in a sequence verified with q) or draws the
// row's token; then it arrives for the sequence, and the last of its dn[b]
// drafted rows runs the accept epilogue (wave 0) -- for a sequence verified
// with q, the residual launch closes it instead.  Every thread of the
// work-group calls this together; all of them continue afterwards.
template <bool kCommit>
__device__ void row_done(const StepParams &p, int b, int r, int dnb, uint32_t units,
                         uint32_t expected, bool spec, Shared &sh) {
    const int tid = threadIdx.x;
    __builtin_amdgcn_s_waitcnt(0);  // this wave's chunk sums are out
    __syncthreads();
    uint32_t *rt = &p.ws.rtk[(int64_t)b * p.ws.rtk_stride + r];
    if (tid < 64) {
        const bool last = arrive_n(rt, units, expected);
        if (tid == 0)
            sh.pick.last = last ? 1 : 0;
    }
    __syncthreads();
    const bool last = sh.pick.last != 0;
    __syncthreads();
    if (!last)
        return;
    if (tid == 0)
        st_u32(rt, 0u);
    if (spec && r < dnb - 1) {
        if (tid < 64)
            spec_test(p, b, r);
    } else {
        // the row's key is not written before pick_row's barrier, so every
        // thread reads the same value and takes the same branch
        unsigned long long *keyp = &p.ws.keys[(int64_t)b * p.ws.key_stride + r];
        float m = 0.0f;
        if (key_max(ld_u64(keyp), m))
            pick_row(p, b, r, m, keyp, sh);
    }
    if (tid < 64 && arrive(&p.ws.tk_all[b * kLineU32], (uint32_t)dnb)) {
        if (spec) {
            st_u32(&p.ws.tk_all[b * kLineU32], 0u);  // the residual launch closes it
        } else {
            final_epilogue<kCommit>(p, b, sh);
            // q row maxima taken before the draft was chosen (the maxima
            // launch's q part) are not used by a copy draft: cleared here
            if (p.qlogits)
                for (int i = tid; i < p.R; i += 64)
                    st_u64(&p.ws.qkeys[(int64_t)b * p.ws.key_stride + i], 0ull);
        }
    }
    __syncthreads();
}

// The polled draw (T > 0, no q, R <= 64): the work-group of row r's first
// segment of the sum launch, once its own sums are stored.  Wave 0 polls the
// row's (chunk, wave) weight sums (each stored + 1, so that 0 is an empty
// slot; the maxima launch zeroed them), then the work-group draws the row's
// token as pick_row does, one vector of the chosen entry per thread.  The
// row's key (the drawn token, or the row maximum's key where nothing is drawn)
// goes to the row's result slot; row 0's work-group keeps its own and, in wave
// 0, polls the other drafted rows' results and runs the accept epilogue.  The
// work-groups of the other segments wait for nothing, and the pollers are the
// first of the grid (segment-major), so every awaited store is made in bounded
// time; the caps guard a broken launch (the error word is set, a row whose
// sums are missing keeps its greedy choice, a missing result counts as none).
// k0 is the row maximum's key as this work-group read it; the key is cleared
// once every work-group of the row has read it (its sums are in).
template <bool kCommit>
__device__ void draw_poller(const StepParams &p, int b, int r, int dn_raw, unsigned long long k0,
                            Shared &sh) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int64_t base = (int64_t)b * p.R;
    unsigned long long *keyp = &p.ws.keys[(int64_t)b * p.ws.key_stride + r];
    unsigned long long *res = p.ws.skeys + (int64_t)b * p.ws.skey_stride;
    const int dnb = clampi(dn_raw, 1, p.R);
    // row 0's draft and lengths, and the row's uniform, requested before the poll
    int tok = -1, par = -1, cL = 0, cdp = 0, cuc = 0;
    unsigned long long uni = 0ull;
    if (wave == 0) {
        if (r == 0) {
            if (lane < p.R) {
                tok = p.dtok[base + lane];
                par = p.dpar ? p.dpar[base + lane] : lane - 1;
            }
            if (kCommit) {
                cL = clampi(p.clen[b], 0, p.Lmax);
                cdp = p.draft_pos[b];
                cuc = p.use_copy[b];
            }
        }
        if (r < dnb)
            uni = p.uniforms[base + r];
    }
    if (r >= dnb) {  // not drawn (no sum work-group of the row reads its key)
        if (tid == 0 && k0)
            st_u64(keyp, 0ull);
        return;
    }
    unsigned long long key = k0 ? k0 : 1ull;  // the result where nothing is drawn
    float m = 0.0f;
    if (!key_max(k0, m)) {
        // one-hot: the other work-groups of the row skip it too (they read the
        // same key, or zero once it is cleared)
        if (tid == 0 && k0)
            st_u64(keyp, 0ull);
    } else {
        if (wave == 0) {
            const int n = p.cpr * kCsumPerChunk;  // <= 256
            const unsigned long long *cs = p.csum + (base + r) * n;
            auto want = [&]() {
                uint32_t w = 0;
                for (int q = 0; q * 64 < n; ++q)
                    if (q * 64 + lane < n)
                        w |= 1u << q;
                return w;
            };
            unsigned long long got[8];
            int rounds = 0;
            const bool ok = poll_wave(cs, n, want, got, p.spin_cap, rounds, [] {});
            if (lane == 0) {
                if (!ok)
                    st_u32(error_word(p, b), 1u);
                sh.draw.ok = ok ? 1 : 0;
            }
            if (ok) {
                // the (chunk, wave) entry holding the target and the target
                // within it (the entry exists, the target being below the
                // total; the clamps only keep every index in range)
                unsigned long long tg;
                int ent;
                if (n <= 64) {
                    // one entry per lane, in index order
                    const unsigned long long x = lane < n ? got[0] - 1ull : 0ull;
                    const unsigned long long inc = wave_scan_u64(x);
                    tg = scaled_target(uni, readlane_u64(inc, 63));
                    ent = __ffsll((long long)__ballot(lane < n && inc > tg)) - 1;
                    ent = ent < 0 ? 0 : ent;
                    tg -= readlane_u64(inc - x, ent);
                } else {
                    // chunk totals, then the waves of the chunk holding the target
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (q * 64 + lane < n)
                            sh.draw.cw[q * 64 + lane] = got[q] - 1ull;
                    unsigned long long cc = 0;
                    if (lane < p.cpr) {
#pragma unroll
                        for (int e = 0; e < kWaves; ++e)
                            cc += sh.draw.cw[lane * kWaves + e];
                    }
                    const unsigned long long inc = wave_scan_u64(cc);
                    tg = scaled_target(uni, readlane_u64(inc, 63));
                    int cst = __ffsll((long long)__ballot(lane < p.cpr && inc > tg)) - 1;
                    cst = cst < 0 ? 0 : cst;
                    tg -= readlane_u64(inc - cc, cst);
                    const unsigned long long ce =
                        lane < kWaves ? sh.draw.cw[cst * kWaves + lane] : 0ull;
                    const unsigned long long ie = wave_scan_u64<3>(ce);
                    int est = __ffsll((long long)__ballot(lane < kWaves && ie > tg)) - 1;
                    est = est < 0 ? 0 : est;
                    tg -= readlane_u64(ie - ce, est);
                    ent = cst * kWaves + est;
                }
                if (lane == 0) {
                    sh.draw.cst = ent / kWaves;
                    sh.draw.est = ent - ent / kWaves * kWaves;
                    sh.draw.tg = tg;
                }
            }
        }
        __syncthreads();
        // every wave has read the row maximum, and every other work-group of
        // the row has (its sums are in): it is cleared
        if (tid == 0)
            st_u64(keyp, 0ull);
        if (sh.draw.ok) {
            // the entry's 256 vectors, vector 64 u + l (block u) in thread 64 u + l;
            // each wave scans its block's weights
            const int cst = sh.draw.cst, est = sh.draw.est;
            const int nq = p.V >> 3;
            const int q0 = cst * kChunkVecs + est * (kUnroll * 64);
            const u32x4 *vp = reinterpret_cast<const u32x4 *>(p.logits + (base + r) * p.V);
            const u32x4 v = q0 + tid < nq ? vp[q0 + tid] : u32x4{0u, 0u, 0u, 0u};
            const unsigned long long w =
                q0 + tid < nq ? (unsigned long long)vec_weight(v, m, p.samp_c) : 0ull;
            const unsigned long long iv = wave_scan_u64(w);
            if (lane == 63)
                sh.draw.bs[wave] = iv;
            __syncthreads();
            // the block holding the target (the same in every wave), then in its
            // wave the vector and the element
            unsigned long long tg = sh.draw.tg, incl = 0;
            int us = kWaves - 1;
            for (int u = 0; u < kWaves; ++u) {
                const unsigned long long bu = sh.draw.bs[u];
                if (tg < incl + bu) {
                    us = u;
                    break;
                }
                incl += bu;
            }
            if (wave == us) {
                tg -= incl;
                int lst = __ffsll((long long)__ballot(iv > tg)) - 1;
                lst = lst < 0 ? 0 : lst;
                tg -= readlane_u64(iv - w, lst);
                // the vector's 8 weights in lanes 0..7, their inclusive prefix
                const int ls = __builtin_amdgcn_readfirstlane(lst);
                const uint32_t x0 = (uint32_t)__builtin_amdgcn_readlane((int)v[0], ls);
                const uint32_t x1 = (uint32_t)__builtin_amdgcn_readlane((int)v[1], ls);
                const uint32_t x2 = (uint32_t)__builtin_amdgcn_readlane((int)v[2], ls);
                const uint32_t x3 = (uint32_t)__builtin_amdgcn_readlane((int)v[3], ls);
                const int wj = (lane >> 1) & 3;
                const uint32_t xj = wj == 0 ? x0 : (wj == 1 ? x1 : (wj == 2 ? x2 : x3));
                unsigned long long ew = 0ull;
                if (lane < 8)
                    ew = (unsigned long long)samp_weight((lane & 1) ? hi_f(xj) : lo_f(xj), m,
                                                         p.samp_c);
                ew = wave_scan_u64<3>(ew);
                int e = __ffsll((long long)__ballot(lane < 8 && ew > tg)) - 1;
                e = e < 0 ? 7 : e;
                const uint32_t y = (uint32_t)(q0 + us * 64 + lst) * 8u + (uint32_t)e;
                if (lane == 0)
                    sh.draw.key = (1ull << 32) | (unsigned long long)(0xFFFFFFFFu - y);
            }
            __syncthreads();
            key = sh.draw.key;
        }
    }
    if (wave != 0)
        return;
    if (r > 0) {
        if (lane == 0)
            st_u64(&res[r], key);
        return;
    }
    // row 0: the other drafted rows' results, then accept, bonus and commit
    unsigned long long kl = lane == 0 ? key : 0ull;
    if (dnb > 1) {
        auto want = [&]() { return lane >= 1 && lane < dnb ? 1u : 0u; };
        unsigned long long got[8];
        int rounds = 0;
        if (!poll_wave(res, dnb, want, got, p.spin_cap, rounds, [] {}) && lane == 0)
            st_u32(error_word(p, b), 1u);
        if (lane >= 1 && lane < dnb) {
            kl = got[0];
            if (got[0])
                st_u64(&res[lane], 0ull);
        }
    }
    const int acc = accept_lanes<kCommit>(p, b, kl > 1ull ? kl : 0ull, tok, par, dn_raw, cL);
    if (kCommit && lane == 0)
        commit_lengths(p, b, cL, cdp, cuc, acc);
}

// Sum launch: work-group (row, segment) adds up the weights of each 16 KB
// chunk of its segment, per wave (a wave's chunk share is < 2^51, exact in
// binary64).  Rows at and beyond dn and rows without a finite maximum are
// skipped.  With the draft's q, a second set of work-groups (after the first
// in the grid) does the same for the q rows that have a drafted child.  With
// the polled draw, the work-group of each row's first segment then draws the
// row's token (draw_poller); else the last one to arrive does (row_done).
template <bool kCommit>
__global__ __launch_bounds__(kThreads) void k_sample_sums(StepParams p) {
    __shared__ Shared sh;
    // segment-major, as the argmax role of the step kernel
    const int nrows = p.B * p.R;
    int idx = blockIdx.x;
    const bool qrow = idx >= nrows * p.segs;
    if (qrow)
        idx -= nrows * p.segs;
    const int s = idx / nrows;
    const int rowi = idx - s * nrows;
    const int b = rowi / p.R, r = rowi - b * p.R;
    const int nq = p.V >> 3;
    // every work-group of the row covers at least one chunk (segs = chunks
    // per row / chunks per work-group, rounded up)
    const int c0 = s * p.seg_chunks;
    const int c1 = c0 + p.seg_chunks < p.cpr ? c0 + p.seg_chunks : p.cpr;
    const u32x4 *vp = reinterpret_cast<const u32x4 *>((qrow ? p.qlogits : p.logits) +
                                                      ((int64_t)b * p.R + r) * p.V);
    u32x4 A[kUnroll], Bv[kUnroll];
    const bool early = p.speculate && !qrow;
    if (early)
        load_chunk_w(A, vp, c0 * kChunkVecs, nq);
    // the draft length and the row maximum requested together (a load the
    // next one waits for would add a round trip); the key is read whether or
    // not the row takes part
    const unsigned long long *keyp =
        &(qrow ? p.ws.qkeys : p.ws.keys)[(int64_t)b * p.ws.key_stride + r];
    const int dn_raw = ld_i32(&p.dn[b]);
    const unsigned long long k_raw = ld_u64(keyp);
    const int dnb = clampi(dn_raw, 1, p.R);
    const bool spec = spec_seq(p, b);
    const bool skip = r >= (qrow ? dnb - 1 : dnb) || (qrow && !spec);  // no part in the draw
    // (the polled draw's first work-group of a skipped row still clears its key)
    const unsigned long long k0 = !skip || (p.draw_poll && s == 0) ? k_raw : 0ull;
    float m = 0.0f;
    bool active = !skip && key_max(k0, m);
    if (p.withhold_seg && p.draw_poll && b == 0 && r == 0 && s == 0)
        active = false;  // test knob: this work-group's sums are never stored
    if (active && !early)
        load_chunk_w(A, vp, c0 * kChunkVecs, nq);
    unsigned long long *cs =
        (qrow ? p.qcsum : p.csum) + ((int64_t)b * p.R + r) * p.cpr * kWaves;
    const unsigned long long mark = p.draw_poll ? 1ull : 0ull;
    for (int c = c0; active && c < c1; ++c) {
        if (c + 1 < c1)
            load_chunk_w(Bv, vp, (c + 1) * kChunkVecs, nq);
        store_block_sums(A, c, nq, m, p.samp_c, cs, mark);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            A[u] = Bv[u];
    }
    if (p.draw_poll) {
        if (s == 0)
            draw_poller<kCommit>(p, b, r, dn_raw, k0, sh);
        return;
    }
    if (skip) {
        __builtin_amdgcn_s_waitcnt(0);
        return;
    }
    // a tested row waits for its p and its q work-groups
    const bool tested = spec && r < dnb - 1;
    row_done<kCommit>(p, b, r, dnb, 1u, (uint32_t)(tested ? 2 * p.segs : p.segs), spec, sh);
}

// Sum launch for long drafts (p.list_mode): the chunks of the drafted rows,
// sequence by sequence and row by row, split evenly over a fixed grid as in
// the streamed verify; a row's maximum is requested together with the
// prefetch of its first chunk.
// The grid is four work-groups per compute unit, all resident at once.
template <bool kCommit>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void
k_sample_sums_stream(StepParams p) {
    __shared__ Shared sh;
    const int lane = threadIdx.x & 63;
    constexpr int Q = kListMaxB / 64;
    const int cpr = p.cpr;
    int first[Q], dnq[Q];
    int carry = 0;
    // (every load issued before any is used: the addresses are clamped rather
    // than the loads made conditional, which would wait for each in turn)
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int b = lane + 64 * q;
        dnq[q] = ld_i32(&p.dn[b < p.B ? b : p.B - 1]);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q)
        dnq[q] = lane + 64 * q < p.B ? clampi(dnq[q], 1, p.R) : 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int cnt = dnq[q] * cpr;
        int inc = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(inc, o);
            if (lane >= o)
                inc += y;
        }
        first[q] = carry + inc - cnt;
        carry += __shfl(inc, 63);
    }
    const int64_t U = carry;
    const int u0 = (int)(U * blockIdx.x / gridDim.x), u1 = (int)(U * (blockIdx.x + 1) / gridDim.x);
    if (u0 >= u1)
        return;
    int b = 0, fb = 0, dnb = 1;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const unsigned long long m = __ballot(lane + 64 * q < p.B && first[q] <= u0);
        if (m) {
            const int l = 63 - __clzll((long long)m);
            b = 64 * q + l;
            fb = __shfl(first[q], l);
            dnb = __shfl(dnq[q], l);
        }
    }
    int r = (u0 - fb) / cpr, c = u0 - fb - r * cpr;
    const int nq = p.V >> 3;
    auto row_vecs = [&](int bb, int rr) {
        return reinterpret_cast<const u32x4 *>(p.logits + ((int64_t)bb * p.R + rr) * p.V);
    };
    u32x4 A[kUnroll], Bv[kUnroll];
    load_chunk_w(A, row_vecs(b, r), c * kChunkVecs, nq);
    unsigned long long key = ld_u64(&p.ws.keys[(int64_t)b * p.ws.key_stride + r]);
    uint32_t done_r = 0;  // units of row (b, r) streamed here
    for (int u = u0; u < u1; ++u) {
        int nb = b, nr = r, nc = c + 1, ndn = dnb;
        if (nc == cpr) {
            nc = 0;
            if (++nr == dnb) {
                nr = 0;
                ++nb;
                if (u + 1 < u1) {
                    const int q = nb >> 6, l = nb & 63;
                    int v = 0;
#pragma unroll
                    for (int qq = 0; qq < Q; ++qq)
                        if (qq == q)
                            v = __shfl(dnq[qq], l);
                    ndn = v;
                }
            }
        }
        unsigned long long nkey = key;
        if (u + 1 < u1) {
            load_chunk_w(Bv, row_vecs(nb, nr), nc * kChunkVecs, nq);
            if (nc == 0)
                nkey = ld_u64(&p.ws.keys[(int64_t)nb * p.ws.key_stride + nr]);
        }
        float m = 0.0f;
        const bool active = key_max(key, m);
        if (active)
            store_block_sums(A, c, nq, m, p.samp_c,
                             p.csum + ((int64_t)b * p.R + r) * cpr * kWaves, 0ull);
        ++done_r;
        if (c == cpr - 1 || u + 1 == u1) {  // end of this row's piece
            row_done<kCommit>(p, b, r, dnb, done_r, (uint32_t)cpr, false, sh);
            done_r = 0;
        }
        b = nb;
        r = nr;
        c = nc;
        dnb = ndn;
        key = nkey;
#pragma unroll
        for (int q = 0; q < kUnroll; ++q)
            A[q] = Bv[q];
    }
}

// Residual weight max(0, P_j Zq - Q_j Zp) of element j, and P_j.
__device__ __forceinline__ u128 resid_weight(float lp, float lq, int j, const SpecRow &s, float c,
                                             unsigned long long &P) {
    P = elem_weight(lp, s.ap, s.mp, j, s.gp, c);
    const unsigned long long Q = elem_weight(lq, s.aq, s.mq, j, s.gq, c);
    const u128 x = (u128)P * s.Zq, y = (u128)Q * s.Zp;
    return x > y ? x - y : (u128)0;
}
// As elem_weight, as a float (an integer below 2^41, exact).
__device__ __forceinline__ float elem_weight_f(float l, bool act, float m, int j, int g, float c) {
    return act ? samp_weight(l, m, c) : (j == g ? 0x1p40f : 0.0f);
}

// The residual weights of the 8 elements of vector q (elements 8q .. 8q+7),
// as sums: over the elements where P Zq > Q Zp, the sums of P (pp) and of Q
// (qp) -- a block's residual sum is then Zq pp - Zp qp, the same integer as
// the sum of its elements' residual weights -- and the sum of every P (ps).
// The products are compared in binary64 (each within 2^-52 of its exact
// value), and in exact 128-bit integers where they lie within 2^-40 of each
// other.  Every sum is an integer below 2^44, exact in binary64.
__device__ __forceinline__ void resid_vec(const u32x4 &vp, const u32x4 &vq, int q,
                                          const SpecRow &s, float c, double zp, double zq,
                                          double &pp, double &qp, double &ps) {
    constexpr double kTie = 1.0 + 0x1p-40;
    auto weights = [&](int e, double &P, double &Q) {
        const uint32_t wp = vp[e >> 1], wq = vq[e >> 1];
        const int j = 8 * q + e;
        P = elem_weight_f((e & 1) ? hi_f(wp) : lo_f(wp), s.ap, s.mp, j, s.gp, c);
        Q = elem_weight_f((e & 1) ? hi_f(wq) : lo_f(wq), s.aq, s.mq, j, s.gq, c);
    };
    uint32_t tie = 0;  // elements whose products lie within the rounding
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        double P, Q;
        weights(e, P, Q);
        const double x = P * zq, y = Q * zp;
        const bool pos = x > y * kTie;
        tie |= (!pos && P != 0.0 && !(y > x * kTie)) ? 1u << e : 0u;
        pp += pos ? P : 0.0;
        qp += pos ? Q : 0.0;
        ps += P;
    }
    if (__any(tie != 0u)) {  // rare (q = p, for one): those elements exactly
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            double P, Q;
            weights(e, P, Q);
            if (((tie >> e) & 1u) &&
                (u128)(unsigned long long)P * s.Zq > (u128)(unsigned long long)Q * s.Zp) {
                pp += P;
                qp += Q;
            }
        }
    }
}

// The residual launch's entries: per block of 64 vectors of the rejected row
// (16 blocks per 16 KB chunk, in index order), its residual sum (128-bit) and
// its P sum.
constexpr int kResBlocks = kChunkVecs / 64;
__device__ __forceinline__ unsigned long long *resid_entry(const StepParams &p, int b, int e) {
    return p.rcsum + ((int64_t)b * p.cpr * kResBlocks + e) * 4;
}
__device__ __forceinline__ u128 entry_value(const unsigned long long *en, bool use_p) {
    const auto ld = [](const unsigned long long *q) {
        return __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    if (use_p)
        return (u128)ld(&en[2]);
    return ((u128)ld(&en[1]) << 64) | ld(&en[0]);
}

// The row's maxima and greedy choices (keys), with the sums Zp and Zq that
// its accept test stored.
__device__ void spec_row_load(const StepParams &p, int b, int r, SpecRow &s) {
    const unsigned long long kp = ld_u64(&p.ws.keys[(int64_t)b * p.ws.key_stride + r]);
    const unsigned long long kq = ld_u64(&p.ws.qkeys[(int64_t)b * p.ws.key_stride + r]);
    const int64_t row = (int64_t)b * p.R + r;
    s.mp = s.mq = 0.0f;
    s.ap = key_max(kp, s.mp);
    s.aq = key_max(kq, s.mq);
    s.gp = decode_key(kp);
    s.gq = decode_key(kq);
    s.Zp = __hip_atomic_load(&p.rz[2 * row], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s.Zq = __hip_atomic_load(&p.rz[2 * row + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The draw after a rejection at row a (wave 0): the blocks' residual sums
// give S and the target floor(u S / 2^64); the block (read in one round trip,
// four per lane, up to 256 blocks; beyond that the chunk of 16 blocks first,
// then its block), the vector (one per lane, p and q read again) and the
// element follow by prefix sums.  With S = 0 (no residual mass) the same
// search runs over the blocks' P sums: the draw from p.  Returns the token in
// every lane.
__device__ int resid_draw(const StepParams &p, int b, int a, const SpecRow &sr) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)b * p.R + a;
    const unsigned long long uni = p.uniforms[row];  // requested with the entries
    const int nb = p.cpr * kResBlocks;                // the row's blocks of 64 vectors
    // (the chunk, the block and the vector exist, the target being below the
    // total; the clamps only keep every index in range)
    u128 tg;
    int blk;  // the block holding the target
    bool use_p;
    if (nb <= 4 * 64) {
        // every block's sum in one round trip, blocks 4 l .. 4 l + 3 in lane l
        auto load4 = [&](bool from_p, u128 (&e4)[4]) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int e = 4 * lane + k;
                e4[k] = e < nb ? entry_value(resid_entry(p, b, e), from_p) : (u128)0;
            }
        };
        u128 e4[4];
        load4(false, e4);
        u128 ls = e4[0] + e4[1] + e4[2] + e4[3];
        u128 inc = wave_scan_u128(ls);
        u128 S = readlane_u128(inc, 63);
        use_p = S == 0;
        if (use_p) {
            load4(true, e4);
            ls = e4[0] + e4[1] + e4[2] + e4[3];
            inc = wave_scan_u128(ls);
            S = readlane_u128(inc, 63);
        }
        tg = mulhi_128_64(S, uni);
        int l = __ffsll((long long)__ballot(inc > tg)) - 1;
        l = l < 0 ? 0 : l;
        tg -= readlane_u128(inc - ls, l);
        // lane l's four blocks, in order
        int k = 3;
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const u128 v = readlane_u128(e4[j], l);
            if (k == 3 && tg < v)
                k = j;
            else if (k == 3)
                tg -= v;
        }
        blk = 4 * l + k;
    } else {
        // chunk totals (16 blocks each), then the blocks of the chunk holding
        // the target: two round trips
        auto chunk_total = [&](bool from_p) -> u128 {
            u128 cc = 0;
            if (lane < p.cpr)
                for (int e = 0; e < kResBlocks; ++e)
                    cc += entry_value(resid_entry(p, b, lane * kResBlocks + e), from_p);
            return cc;
        };
        u128 cc = chunk_total(false);
        u128 inc = wave_scan_u128(cc);
        u128 S = readlane_u128(inc, 63);
        use_p = S == 0;
        if (use_p) {
            cc = chunk_total(true);
            inc = wave_scan_u128(cc);
            S = readlane_u128(inc, 63);
        }
        tg = mulhi_128_64(S, uni);
        int cst = __ffsll((long long)__ballot(lane < p.cpr && inc > tg)) - 1;
        cst = cst < 0 ? 0 : cst;
        tg -= readlane_u128(inc - cc, cst);
        const u128 ce =
            lane < kResBlocks ? entry_value(resid_entry(p, b, cst * kResBlocks + lane), use_p) : 0;
        const u128 ie = wave_scan_u128<4>(ce);  // lanes 0..15
        int est = __ffsll((long long)__ballot(lane < kResBlocks && ie > tg)) - 1;
        est = est < 0 ? 0 : est;
        tg -= readlane_u128(ie - ce, est);
        blk = cst * kResBlocks + est;
    }
    // the block's 64 vectors, one per lane
    const int nq = p.V >> 3;
    const int q = blk * 64 + lane;
    const u32x4 *pv = reinterpret_cast<const u32x4 *>(p.logits + row * p.V);
    const u32x4 *qv = reinterpret_cast<const u32x4 *>(p.qlogits + row * p.V);
    u32x4 xp = u32x4{0u, 0u, 0u, 0u}, xq = u32x4{0u, 0u, 0u, 0u};
    u128 w = 0;
    if (q < nq) {
        xp = pv[q];
        xq = qv[q];
        double pp = 0.0, qp = 0.0, ps = 0.0;
        resid_vec(xp, xq, q, sr, p.samp_c, (double)sr.Zp, (double)sr.Zq, pp, qp, ps);
        w = use_p ? (u128)(unsigned long long)ps
                  : (u128)(unsigned long long)pp * sr.Zq - (u128)(unsigned long long)qp * sr.Zp;
    }
    const u128 iv = wave_scan_u128(w);
    int lst = __ffsll((long long)__ballot(iv > tg)) - 1;
    lst = lst < 0 ? 0 : lst;
    tg -= readlane_u128(iv - w, lst);
    // that vector's 8 weights in lanes 0..7, their inclusive prefix
    const int ls = __builtin_amdgcn_readfirstlane(lst);
    const int wj = (lane >> 1) & 3;
    uint32_t hp = 0, hq = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t xpk = (uint32_t)__builtin_amdgcn_readlane((int)xp[k], ls);
        const uint32_t xqk = (uint32_t)__builtin_amdgcn_readlane((int)xq[k], ls);
        hp = wj == k ? xpk : hp;
        hq = wj == k ? xqk : hq;
    }
    const int qs = blk * 64 + ls;
    u128 ew = 0;
    if (lane < 8) {
        unsigned long long P;
        const u128 r = resid_weight((lane & 1) ? hi_f(hp) : lo_f(hp),
                                    (lane & 1) ? hi_f(hq) : lo_f(hq), 8 * qs + lane, sr, p.samp_c,
                                    P);
        ew = use_p ? (u128)P : r;
    }
    ew = wave_scan_u128<3>(ew);
    int e = __ffsll((long long)__ballot(lane < 8 && ew > tg)) - 1;
    e = e < 0 ? 7 : e;
    return 8 * qs + e;
}
// Outputs of a sequence verified with q: accepted prefix a, then the emitted
// token (bonus).  dt: lane i's drafted token i + 1 (i < 64), read before the
// draw; cL: the context length (decode loop).
template <bool kCommit>
__device__ void spec_epilogue(const StepParams &p, int b, int a, int bonus, int dt, int cL) {
    const int lane = threadIdx.x & 63;
    const int64_t base = (int64_t)b * p.R;
    for (int i = lane; i < p.R; i += 64) {
        const int v =
            i < a ? (i < 64 ? dt : ld_i32(&p.dtok[base + i + 1])) : (i == a ? bonus : -1);
        p.out_tokens[base + i] = v;
        if (p.amax)
            p.amax[base + i] = v;
        if (kCommit && i <= a && cL + i < p.Lmax)
            p.ctok[(int64_t)b * p.Lmax + cL + i] = v;
        st_u64(&p.ws.keys[(int64_t)b * p.ws.key_stride + i], 0ull);
        st_u64(&p.ws.qkeys[(int64_t)b * p.ws.key_stride + i], 0ull);
    }
    if (lane == 0) {
        p.accept_len[b] = a;
        p.accept_node[b] = a;
        p.bonus[b] = bonus;
        if (kCommit) {  // a neural step: the draft model drafted the accepted tokens
            const int Lnew = cL + a + 1 < p.Lmax ? cL + a + 1 : p.Lmax;
            const int pos = clampi(cL + a, 0, Lnew);
            p.clen[b] = Lnew;
            p.draft_pos[b] = pos;
            p.lag[b] = Lnew - pos;
        }
    }
}

// Residual launch of sequences verified with q: work-group (unit s, sequence
// b), unit-major; unit s covers blocks 8 s .. 8 s + 7 of 64 vectors (two per
// wave, one vector per lane each, both requested together).  Every
// work-group finds the first rejected row a from the tests; if there is one,
// each wave adds up its blocks' residual weights (128-bit, through resid_vec's
// sums) and P weights.
// (Two blocks per wave keep the grid within the resident work-groups, 1024
// for C2: one block per wave ran the 2048 work-groups in two batches, C2 at
// T = 0.7 with q 81.9 us per step against 80.0.)  The last of the sequence's rsegs
// work-groups draws the emitted token (the residual draw at a, or the bonus
// drawn from p at the last row when every test passed) and writes the
// outputs.
template <bool kCommit>
__global__ __launch_bounds__(kThreads) void k_spec_residual(StepParams p) {
    const int s = blockIdx.x / p.B, b = blockIdx.x - s * p.B;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    // whether the sequence was verified with q, its draft length and the
    // first 64 rows' tests, requested together: unconditional loads (a load
    // under a branch, or into a register a later address reuses, would be
    // waited for before the next is issued)
    const int32_t *cp = p.spec_copy ? &p.spec_copy[b] : &p.dn[b];
    const int copy_raw = ld_i32(cp);
    const int dn_raw = ld_i32(&p.dn[b]);
    const uint32_t dec_raw = __hip_atomic_load(
        &p.rdec[(int64_t)b * p.R + (lane < p.R ? lane : p.R - 1)], __ATOMIC_RELAXED,
        __HIP_MEMORY_SCOPE_AGENT);
    const int copy = p.spec_copy ? copy_raw : 0;
    const uint32_t dec0 = lane < p.R ? dec_raw : 1u;
    if (!p.qlogits || copy != 0)  // not verified with q (spec_seq)
        return;
    const int dnb = clampi(dn_raw, 1, p.R);
    int a = dnb - 1;
    for (int r0 = 0; r0 < dnb - 1; r0 += 64) {
        const int r = r0 + lane;
        const bool rej = r < dnb - 1 &&
                         (r0 == 0 ? dec0
                                  : __hip_atomic_load(&p.rdec[(int64_t)b * p.R + r],
                                                      __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)) != 1u;
        const unsigned long long m = __ballot(rej);
        if (m) {
            a = r0 + __ffsll((long long)m) - 1;
            break;
        }
    }
    const bool resid = a < dnb - 1;
    SpecRow sr;
    if (resid) {
        spec_row_load(p, b, a, sr);
        const int nq = p.V >> 3;
        const int64_t row = (int64_t)b * p.R + a;
        u32x4 vp[2], vq[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int q = ((s * kWaves + wave) * 2 + h) * 64 + lane;
            const int qc = q < nq ? q : nq - 1;
            vp[h] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4 *>(p.logits + row * p.V) + qc);
            vq[h] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4 *>(p.qlogits + row * p.V) + qc);
        }
        const double zp = (double)sr.Zp, zq = (double)sr.Zq;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int blk = (s * kWaves + wave) * 2 + h;
            const int q = blk * 64 + lane;
            double pp = 0.0, qp = 0.0, psd = 0.0;
            if (q < nq)
                resid_vec(vp[h], vq[h], q, sr, p.samp_c, zp, zq, pp, qp, psd);
            // (the block's sums are below 2^50: exact in binary64)
            const unsigned long long PP = (unsigned long long)wave_sum_f64(pp);
            const unsigned long long QP = (unsigned long long)wave_sum_f64(qp);
            const unsigned long long ps = (unsigned long long)wave_sum_f64(psd);
            const u128 acc = (u128)PP * sr.Zq - (u128)QP * sr.Zp;
            if (lane == 0 && blk < p.cpr * kResBlocks) {
                unsigned long long *en = resid_entry(p, b, blk);
                __hip_atomic_store(&en[0], (unsigned long long)acc, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&en[1], (unsigned long long)(acc >> 64), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&en[2], ps, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid >= 64)
        return;
    if (arrive(&p.ws.tk_all[b * kLineU32], (uint32_t)p.rsegs)) {
        if (lane == 0)
            st_u32(&p.ws.tk_all[b * kLineU32], 0u);
        // the epilogue's reads, requested before the draw's
        const int dt = lane + 1 < p.R ? ld_i32(&p.dtok[(int64_t)b * p.R + lane + 1]) : -1;
        const int cL = kCommit ? clampi(p.clen[b], 0, p.Lmax) : 0;
        const int bonus = resid ? resid_draw(p, b, a, sr)
                                : decode_key(ld_u64(&p.ws.keys[(int64_t)b * p.ws.key_stride +
                                                               dnb - 1]));
        spec_epilogue<kCommit>(p, b, a, bonus, dt, cL);
    }
}

// ------------------------------------------------------------- copy-mode labels

// Copy-mode labels for probe training (Sec. 3.2, Problem Formulation):
// position j is copy-mode iff an n-token window covering it repeats an
// earlier window, i.e. the window starting at some s in [j - n + 1, j] is not
// the first occurrence of its n tokens.  An open-addressing table per
// sequence (linear probing, at most a quarter full) holds one slot per distinct
// window content with the complement of its earliest start (0: empty):
// k_label_insert claims a slot with a compare-and-swap or, when the slot's
// window has the same tokens (compared token by token, never by hash),
// lowers its start with an atomic max of the complement; k_label_write then
// marks the starts s whose slot holds an earlier start and widens them into
// labels, and k_label_clear empties the table.  The hash only spreads
// the windows over the table: the result does not depend on it.  All windows
// of one content walk the same probe sequence, and a slot never empties or
// changes content, so each content ends in exactly one slot and every walk
// reaches it before any empty slot.

// Windows are read 8 tokens at a time, the 8 loads of a group issued together
// (one memory round trip per group rather than per token).
constexpr int kWinGroup = 8;

// Slot of the window at s: a multiplicative mix of its tokens.
__device__ __forceinline__ uint32_t label_hash(const int32_t *x, int s, int n) {
    uint32_t h = 0x9E3779B9u;
    for (int i0 = 0; i0 < n; i0 += kWinGroup) {
        int32_t t[kWinGroup];
#pragma unroll
        for (int i = 0; i < kWinGroup; ++i)
            t[i] = i0 + i < n ? x[s + i0 + i] : 0;
#pragma unroll
        for (int i = 0; i < kWinGroup; ++i)
            if (i0 + i < n) {
                h = (h ^ (uint32_t)t[i]) * 0x85EBCA6Bu;
                h ^= h >> 15;
            }
    }
    h *= 0xC2B2AE35u;
    return h ^ (h >> 16);
}

__device__ __forceinline__ bool same_window(const int32_t *x, int s1, int s2, int n) {
    for (int i0 = 0; i0 < n; i0 += kWinGroup) {
        int32_t a[kWinGroup], c[kWinGroup];
#pragma unroll
        for (int i = 0; i < kWinGroup; ++i) {
            a[i] = i0 + i < n ? x[s1 + i0 + i] : 0;
            c[i] = i0 + i < n ? x[s2 + i0 + i] : 0;
        }
        bool eq = true;
#pragma unroll
        for (int i = 0; i < kWinGroup; ++i)
            eq = eq && a[i] == c[i];
        if (!eq)
            return false;
    }
    return true;
}

// One lane per window start s <= L - n of sequence b.
__global__ __launch_bounds__(kThreads) void k_label_insert(StepParams p, int32_t n, int32_t tsize,
                                                           uint32_t *table) {
    const int per = (p.Lmax + kThreads - 1) / kThreads;
    const int b = blockIdx.x / per;
    const int s = (blockIdx.x - b * per) * kThreads + (int)threadIdx.x;
    const int L = clampi(p.lengths[b], 0, p.Lmax);
    if (s > L - n)
        return;
    const int32_t *x = p.tokens + (int64_t)b * p.Lmax;
    uint32_t *tab = table + (int64_t)b * tsize;
    const uint32_t mask = (uint32_t)tsize - 1u;
    uint32_t slot = label_hash(x, s, n) & mask;
    const uint32_t mine = ~(uint32_t)s;
    for (int probe = 0; probe < tsize; ++probe) {
        // one compare-and-swap claims an empty slot or returns its start (a
        // plain read first costs one more round trip for every first window)
        const uint32_t cur = atomicCAS(&tab[slot], 0u, mine);
        if (cur == 0u)
            return;  // first of its content to arrive here
        if (same_window(x, (int)~cur, s, n)) {
            if (cur < mine)  // a later start is there: the earliest one wins
                atomicMax(&tab[slot], mine);
            return;
        }
        slot = (slot + 1u) & mask;
    }
}

// Whether the window at s (s <= L - n) repeats an earlier one: its content's
// slot holds a start < s.
__device__ __forceinline__ bool label_repeats(const int32_t *x, const uint32_t *tab,
                                              uint32_t mask, int s, int n) {
    uint32_t slot = label_hash(x, s, n) & mask;
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        const uint32_t cur = tab[slot];
        if (cur == 0u)
            return false;  // unreachable: the window's own insert filled a slot first
        if (same_window(x, (int)~cur, s, n))
            return (int)~cur < s;
        slot = (slot + 1u) & mask;
    }
    return false;
}

// Labels of 256 positions of sequence b (one 64-position block per wave of
// the first four): bit l of block w's ballot E_w says whether the window
// starting at 64 w + l repeats an earlier one; position j is copy-mode iff
// such a start lies in [j - n + 1, j], i.e. bit j of E | E << 1 | ... |
// E << (n - 1) with the previous block's bits carried in.  A fifth wave looks
// up the block before the range, so that no wave walks two blocks.
constexpr int kLabelWriteThreads = kThreads + 64;
__global__ __launch_bounds__(kLabelWriteThreads) void k_label_write(StepParams p, int32_t n,
                                                                    int32_t tsize,
                                                                    const uint32_t *table,
                                                                    uint8_t *labels) {
    __shared__ unsigned long long E[kWaves + 1];  // E[0]: the block before the range
    const int per = (p.Lmax + kThreads - 1) / kThreads;
    const int b = blockIdx.x / per;
    const int g = blockIdx.x - b * per;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int L = clampi(p.lengths[b], 0, p.Lmax);
    const int32_t *x = p.tokens + (int64_t)b * p.Lmax;
    const uint32_t *tab = table + (int64_t)b * tsize;
    const uint32_t mask = (uint32_t)tsize - 1u;
    // waves 0..3: starts 256 g + tid; wave 4: the 64 starts before them
    const int s = wave < kWaves ? g * kThreads + tid : g * kThreads - 64 + lane;
    const unsigned long long m =
        __ballot(s >= 0 && s <= L - n && label_repeats(x, tab, mask, s, n));
    if (lane == 0)
        E[wave < kWaves ? wave + 1 : 0] = m;
    __syncthreads();
    if (wave == kWaves)
        return;
    const unsigned long long Ec = E[wave + 1], Ep = E[wave];
    unsigned long long Y = Ec;
    for (int u = 1; u < n; ++u)
        Y |= (Ec << u) | (Ep >> (64 - u));
    if (s < p.Lmax)
        labels[(int64_t)b * p.Lmax + s] = (uint8_t)((Y >> lane) & 1ull);
}

// Empties the window tables again (after every lookup has finished); the
// tables are 256-byte aligned and a whole number of 16-byte vectors.
__global__ __launch_bounds__(kThreads) void k_label_clear(u32x4 *table, int64_t vecs) {
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < vecs;
         i += (int64_t)gridDim.x * kThreads)
        table[i] = u32x4{0u, 0u, 0u, 0u};
}

// ------------------------------------------------------------- kernels

// The row an argmax work-group of the fused step (block index blk) takes among
// the nrows rows of its segment (rowi0: its place in the segment's run of
// work-groups).  Work-groups go to the 8 XCDs in turn (block index mod 8);
// when nrows is a multiple of 8 this gives each XCD a contiguous eighth of the
// rows (and, when B is too, whole sequences).  Measured against every eighth
// row per XCD, same box: C3 28.69 -> 28.54 us, C4 10.34 -> 10.19 us, C2
// 15.11 -> 15.07 us.  The polling verify launch keeps every eighth row per
// XCD: there the contiguous split made C5 (2.7 GB of rows) 408 -> 428 us.
__device__ __forceinline__ int xcd_row(int blk, int rowi0, int nrows) {
    return (nrows & 7) == 0 ? (blk & 7) * (nrows >> 3) + (rowi0 >> 3) : rowi0;
}

// kQ: the row maxima launch before a draw at T > 0 that also takes the
// draft's q rows (qmax; compiled apart, so that the other launches keep their
// code).
template <bool kMulti, bool kCommit, bool kQ = false>
__global__ __launch_bounds__(kThreads) void k_switchsd(StepParams p) {
    TL_MARK(0);
    // the argmax role's kept chunks share the union: the role is over (every
    // wave) before an epilogue of this work-group uses LDS
    __shared__ Shared sh;
    const int blk = blockIdx.x;
    int b, t = 0;
    int role;  // 0 scan, 1 stand-alone probe, 2 argmax
    Prefetch pre = {1, -1, -1};
    // block order: [probe work-groups | scan tiles | argmax segments]
    const int n_probe = p.n_front_wg - p.n_scan_wg;
    if (blk < n_probe) {
        b = blk;
        probe_role(p, b, sh);
        role = 1;
    } else if (blk < p.n_front_wg) {
        b = (blk - n_probe) / p.scan_tiles;
        t = blk - n_probe - b * p.scan_tiles;
        scan_role<kMulti>(p, b, t, sh, pre);
        role = 0;
    } else {
        // segment-major: the first B * R work-groups take every row's first
        // segment, the next B * R the second ...  Work-groups later in the
        // dispatch stream more slowly (they share their CUs with ones issued
        // earlier), and a sequence waits for its slowest segment; so every
        // sequence gets segments from the whole dispatch order.
        // (with qmax, the same again over the draft's logits after them)
        const int idx0 = blk - p.n_front_wg;
        const int nrows = p.B * p.R;
        const bool qpart = kQ && idx0 >= nrows * p.segs;
        const int idx = qpart ? idx0 - nrows * p.segs : idx0;
        const int s = idx / nrows;
        const int rowi = xcd_row(blk, idx - s * nrows, nrows);
        b = rowi / p.R;
        argmax_role(p, b, rowi - b * p.R, s, sh, sh.am.keep, qpart);
        role = 2;
    }
    TL_MARK(1);
    TL_TAG(((unsigned long long)role << 32) | (uint32_t)b);
    if (threadIdx.x >= 64)
        return;  // waves 1.. are done; wave 0 arrives and may run an epilogue
    if (role == 0 && p.epi_front != EPI_NONE) {
        // The scan's reads, the prefetched neural draft included, returned
        // long ago; an explicit wait for them here costs nothing and keeps the
        // compiler's count of outstanding reads exact through the branches
        // below (otherwise a use of the prefetched values after them waits for
        // every store of the front as well).
        __builtin_amdgcn_s_waitcnt(0);
        DraftRegs dr = {-1, -1, 1, 0, 1, 0, -1, 0, -1, 0.0f, 0u, false, false, false};
        bool chose = false;  // this work-group chose sequence b's draft
        if (p.scan_tiles == 1) {
            front_local(p, b, sh, pre, dr);
            chose = true;
            TL_MARK(2);
        } else {
            const int lane = threadIdx.x;
            const bool fread = p.epi_front == EPI_SELECT && p.probe_on;
            if (t == 0 && p.scan_probe && lane == 0)
                st_f32(&p.z[b], probe_combine(sh.scan.ps, sh.scan.pc, p.bias));
            if (p.poll_front) {
                if (kMulti && p.W > 1) {
                    // every tile's W most recent ends per length go to its lists
                    // first (the chooser reads them once the slots are in); a
                    // tile's slot store follows the completed list stores
                    int32_t *cb = p.ws.cand + (int64_t)b * p.ws.cand_stride +
                                  (int64_t)t * SWITCHSD_MAX_NGRAM * p.W;
                    for (int j = 0; j < p.n_ngram; ++j) {
                        const int v = merge_waves(p, sh, j);
                        if (lane < p.W)
                            st_i32(&cb[j * p.W + lane], v);
                    }
                    __builtin_amdgcn_s_waitcnt(0);
                }
                if (t + 1 < p.scan_tiles) {
                    // this tile's result in its own slots; nothing waits here
                    // (the test knob withholds sequence 0's first tile)
                    if (lane < p.n_ngram && !(p.withhold_seg && b == 0 && t == 0))
                        st_i32(&p.ws.tslot[(int64_t)b * p.ws.tslot_stride +
                                           t * SWITCHSD_MAX_NGRAM + lane],
                               sh.scan.red[lane] + 1);
                } else {
                    // the probe's flag is read once with the tiles' slots
                    const uint32_t fl0 = fread ? ld_u32(probe_flag(p, b)) : 0u;
                    const int32_t sl = poll_tiles(p, b, sh, dr);
                    front_remote(p, b, t, sh, pre, dr, sl, fl0);
                    chose = true;
                    TL_MARK(2);
                }
            } else {
                if (lane < p.n_ngram && sh.scan.red[lane] > 0)
                    atomicMax(&p.ws.mslot[b * kLineU32 + lane], sh.scan.red[lane]);
                if (kMulti && p.W > 1) {
                    int32_t *cb = p.ws.cand + (int64_t)b * p.ws.cand_stride +
                                  (int64_t)t * SWITCHSD_MAX_NGRAM * p.W;
                    for (int j = 0; j < p.n_ngram; ++j) {
                        const int v = merge_waves(p, sh, j);
                        if (lane < p.W)
                            st_i32(&cb[j * p.W + lane], v);
                    }
                }
                if (arrive(&p.ws.tk_front[b * kLineU32], p.exp_front)) {
                    // the tiles' results and the probe's flag, requested together
                    const uint32_t fl0 = fread ? ld_u32(probe_flag(p, b)) : 0u;
                    int32_t sl = 0;
                    if (lane < p.n_ngram) {
                        sl = ld_i32(&p.ws.mslot[b * kLineU32 + lane]);
                        st_i32(&p.ws.mslot[b * kLineU32 + lane], 0);
                    }
                    front_remote(p, b, t, sh, pre, dr, sl, fl0);
                    chose = true;
                    TL_MARK(2);
                }
            }
        }
        // (polling is compiled into the one-candidate kernels only: the host
        // never sets it for several candidates, and the several-candidate
        // kernels then stay small enough for the accept epilogue to be inlined)
        if (!kMulti && p.poll_accept && chose) {
            poll_epilogue<kCommit>(p, b, dr, sh);
#ifdef SWITCHSD_TIMELINE
            __builtin_amdgcn_s_waitcnt(0);
#endif
            TL_MARK(4);
        }
    }
    if (!kMulti && p.poll_accept)
        return;  // an argmax work-group's slot is its only hand-off
    if (p.epi_accept && role != 1) {
        const bool last = arrive(&p.ws.tk_all[b * kLineU32], p.exp_all);
        TL_MARK(3);
        if (last) {
            final_epilogue<kCommit>(p, b, sh);
#ifdef SWITCHSD_TIMELINE
            __builtin_amdgcn_s_waitcnt(0);
#endif
            TL_MARK(4);
        }
    }
}

// The verify launch with polling (T = 0, R <= 64, B no larger than the CU
// count): block order [one poller per sequence | argmax row segments,
// segment-major].  A poller holds its sequence's draft and runs the accept
// epilogue once the segment results are in (poll_epilogue); the argmax
// work-groups store their results and wait for nothing.
template <bool kCommit>
__global__ __launch_bounds__(kThreads) void k_verify_poll(StepParams p) {
    __shared__ Shared sh;
    if ((int)blockIdx.x < p.B) {
        if (threadIdx.x < 64) {
            DraftRegs dr = {-1, -1, 1, 0, 1, 0, -1, 0, -1, 0.0f, 0u, false, false, false};
            poller_draft<kCommit>(p, (int)blockIdx.x, dr);
            poll_epilogue<kCommit>(p, (int)blockIdx.x, dr, sh);
        }
        return;
    }
    const int idx = (int)blockIdx.x - p.B;
    const int nrows = p.B * p.R;
    const int s = idx / nrows;
    const int rowi = idx - s * nrows;  // (every eighth row per XCD: see xcd_row)
    const int b = rowi / p.R;
    argmax_role(p, b, rowi - b * p.R, s, sh, sh.am.keep);
}

// The grid is four work-groups per compute unit, all resident at once.
template <bool kCommit>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void
k_verify_stream(StepParams p) {
    __shared__ Shared sh;
    __shared__ u32x4 keep[kChunkVecs];  // each lane's kept chunk (running argmax)
    verify_stream<kCommit>(p, sh, keep);
}

// Stand-alone commit of a finished step (one wave per sequence).
__global__ __launch_bounds__(64) void k_commit(StepParams p) {
    const int b = blockIdx.x, lane = threadIdx.x;
    const int L = clampi(p.clen[b], 0, p.Lmax);
    const int a = clampi(p.accept_len[b], 0, p.R - 1);
    const int Lnew = L + a + 1 < p.Lmax ? L + a + 1 : p.Lmax;
    for (int j = lane; L + j < Lnew; j += 64)
        p.ctok[(int64_t)b * p.Lmax + L + j] = p.out_tokens[(int64_t)b * p.R + j];
    if (lane == 0) {
        const int pos = clampi(p.use_copy[b] ? p.draft_pos[b] : L + a, 0, Lnew);
        p.clen[b] = Lnew;
        p.draft_pos[b] = pos;
        p.lag[b] = Lnew - pos;
    }
}

// Reads and clears the error words of B sequences (one work-group, any B).
__global__ __launch_bounds__(kThreads) void k_status(int32_t *mslot, int32_t B, int32_t *out) {
    int err = 0;
    for (int b = threadIdx.x; b < B; b += kThreads) {
        uint32_t *w = (uint32_t *)&mslot[(int64_t)b * kLineU32 + kLineU32 - 2];
        if (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) {
            err = 1;
            st_u32(w, 0u);
        }
    }
    err = __syncthreads_or(err);
    if (threadIdx.x == 0)
        out[0] = err ? SWITCHSD_EDEVICE : SWITCHSD_OK;
}

__global__ __launch_bounds__(64) void k_select(StepParams p) {
    __shared__ ChainShared ch;
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int cl = lane < p.W ? clampi(p.copy_len_in[(int64_t)b * p.W + lane], 0, p.k) : 0;
    const int total = chain_layout(p, cl, ch);
    const int use = (p.match_n_in[b] >= p.kappa) && (p.z_in[b] >= p.theta);
    const int32_t *ct = p.copy_tokens_in + (int64_t)b * p.W * p.k;
    const int64_t base = (int64_t)b * p.R;
    DraftRegs dr;
    write_chains(p, b, use, total, clampi(p.nn[b], 1, p.R), ch,
                 [&](int c, int j) { return ct[c * p.k + j]; },
                 [&](int i, int &tok, int &par) {
                     tok = p.ntok[base + i];
                     par = p.npar ? p.npar[base + i] : i - 1;
                 },
                 dr);
}

// One work-group of 256 (row, word) cells of sequence b's ancestor mask;
// dpar of the sequence staged in LDS.  A cell walks its row's path from the
// node up and keeps the ancestors that fall into its word; indices fall
// along the path, so the walk stops below the word.
__global__ __launch_bounds__(kThreads) void k_tree_mask(const int32_t *dpar, const int32_t *dn,
                                                        int32_t R, int32_t words,
                                                        int32_t blocks_per_seq,
                                                        uint32_t *mask) {
    __shared__ int32_t par[SWITCHSD_MAX_R];
    const int b = blockIdx.x / blocks_per_seq;
    const int blk = blockIdx.x - b * blocks_per_seq;
    const int tid = threadIdx.x;
    for (int i = tid; i < R; i += kThreads)
        par[i] = dpar ? dpar[(int64_t)b * R + i] : i - 1;
    __syncthreads();
    const int cell = blk * kThreads + tid;
    if (cell >= R * words)
        return;
    const int i = cell / words, w = cell - i * words;
    const int dnb = clampi(dn[b], 0, R);
    uint32_t acc = 0u;
    if (i < dnb && i >= 32 * w) {
        int node = i;
        for (;;) {
            if ((node >> 5) == w)
                acc |= 1u << (node & 31);
            if (node == 0)
                break;
            const int q = par[node];
            if (q < 0 || q >= node)
                break;
            node = q;
            if (node < 32 * w)
                break;
        }
    }
    mask[(int64_t)b * R * words + cell] = acc;
}

}  // namespace

int launch_tree_mask_kernel(const int32_t *dpar, const int32_t *dn, int32_t B, int32_t R,
                            uint32_t *mask, hipStream_t stream) {
    const int32_t words = (R + 31) / 32;
    const int32_t per = (R * words + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(k_tree_mask, dim3((unsigned)((int64_t)B * per)), dim3(kThreads), 0, stream,
                       dpar, dn, R, words, per, mask);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_step_kernel(const StepParams &p, int64_t grid, hipStream_t stream) {
    if (p.n_poll_wg > 0)
        if (p.commit)
            hipLaunchKernelGGL((k_verify_poll<true>), dim3((unsigned)grid), dim3(kThreads), 0,
                               stream, p);
        else
            hipLaunchKernelGGL((k_verify_poll<false>), dim3((unsigned)grid), dim3(kThreads), 0,
                               stream, p);
    else if (p.list_mode)
        if (p.commit)
            hipLaunchKernelGGL((k_verify_stream<true>), dim3((unsigned)grid), dim3(kThreads), 0,
                               stream, p);
        else
            hipLaunchKernelGGL((k_verify_stream<false>), dim3((unsigned)grid), dim3(kThreads), 0,
                               stream, p);
    else if (p.W > 1 && p.commit)
        hipLaunchKernelGGL((k_switchsd<true, true>), dim3((unsigned)grid), dim3(kThreads), 0,
                           stream, p);
    else if (p.W > 1)
        hipLaunchKernelGGL((k_switchsd<true, false>), dim3((unsigned)grid), dim3(kThreads), 0,
                           stream, p);
    else if (p.qmax && p.commit)
        hipLaunchKernelGGL((k_switchsd<false, true, true>), dim3((unsigned)grid), dim3(kThreads),
                           0, stream, p);
    else if (p.qmax)
        hipLaunchKernelGGL((k_switchsd<false, false, true>), dim3((unsigned)grid),
                           dim3(kThreads), 0, stream, p);
    else if (p.commit)
        hipLaunchKernelGGL((k_switchsd<false, true>), dim3((unsigned)grid), dim3(kThreads), 0,
                           stream, p);
    else
        hipLaunchKernelGGL((k_switchsd<false, false>), dim3((unsigned)grid), dim3(kThreads), 0,
                           stream, p);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_sample_sums_kernel(const StepParams &p, int64_t grid, hipStream_t stream) {
    const dim3 g((unsigned)grid);
    if (p.list_mode && p.commit)
        hipLaunchKernelGGL((k_sample_sums_stream<true>), g, dim3(kThreads), 0, stream, p);
    else if (p.list_mode)
        hipLaunchKernelGGL((k_sample_sums_stream<false>), g, dim3(kThreads), 0, stream, p);
    else if (p.commit)
        hipLaunchKernelGGL((k_sample_sums<true>), g, dim3(kThreads), 0, stream, p);
    else
        hipLaunchKernelGGL((k_sample_sums<false>), g, dim3(kThreads), 0, stream, p);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_spec_residual_kernel(const StepParams &p, int64_t grid, hipStream_t stream) {
    const dim3 g((unsigned)grid);
    if (p.commit)
        hipLaunchKernelGGL((k_spec_residual<true>), g, dim3(kThreads), 0, stream, p);
    else
        hipLaunchKernelGGL((k_spec_residual<false>), g, dim3(kThreads), 0, stream, p);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_status_kernel(int32_t *mslot, int32_t B, int32_t *out, hipStream_t stream) {
    hipLaunchKernelGGL(k_status, dim3(1), dim3(kThreads), 0, stream, mslot, B, out);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_commit_kernel(const StepParams &p, hipStream_t stream) {
    hipLaunchKernelGGL(k_commit, dim3((unsigned)p.B), dim3(64), 0, stream, p);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_label_kernels(const StepParams &p, int32_t n, uint8_t *labels, int32_t tsize,
                         void *table, hipStream_t stream) {
    const int64_t per = (p.Lmax + kThreads - 1) / kThreads;
    const dim3 grid((unsigned)((int64_t)p.B * per));
    hipLaunchKernelGGL(k_label_insert, grid, dim3(kThreads), 0, stream, p, n, tsize,
                       (uint32_t *)table);
    if (hipGetLastError() != hipSuccess)
        return SWITCHSD_EHIP;
    hipLaunchKernelGGL(k_label_write, grid, dim3(kLabelWriteThreads), 0, stream, p, n, tsize,
                       (const uint32_t *)table, labels);
    if (hipGetLastError() != hipSuccess)
        return SWITCHSD_EHIP;
    const int64_t vecs = (int64_t)p.B * tsize / 4;  // tsize is a multiple of 64
    const int64_t cgrid = (vecs + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(k_label_clear, dim3((unsigned)(cgrid < 65536 ? cgrid : 65536)),
                       dim3(kThreads), 0, stream, (u32x4 *)table, vecs);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

int launch_select_kernel(const StepParams &p, hipStream_t stream) {
    hipLaunchKernelGGL(k_select, dim3((unsigned)p.B), dim3(64), 0, stream, p);
    return hipGetLastError() == hipSuccess ? SWITCHSD_OK : SWITCHSD_EHIP;
}

}  // namespace switchsd
