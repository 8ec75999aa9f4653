// switchsd_api.cpp -- C entry points: argument validation, grid layout and
// dispatch of the gfx950 kernels.  Every check runs on the host before any
// HIP call; a rejected call launches nothing.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#include "switchsd.h"
#include "switchsd_internal.h"

using namespace switchsd;

namespace {

constexpr size_t kAlign = 256;

// Test knob (switchsd_test_withhold_probe_flag): the step's probe work-groups
// never set their flag and the front gives up its wait after a few
// iterations, so that the give-up path runs with every kernel exiting.
std::atomic<int> g_withhold_probe_flag{0};
// Test knob (switchsd_test_withhold_segment): in the fused step, sequence 0's
// row 0 segment 0 and (with 2..64 scan tiles) its scan tile 0 never store
// their results, and the accept epilogue's and the last tile's polls give up
// after a few iterations.
std::atomic<int> g_withhold_segment{0};

#ifdef SWITCHSD_TIMELINE
// Timeline build only: the buffer of the next step launches' phase stamps
// (8 per work-group), set by switchsd_timeline_buffer.
std::atomic<unsigned long long *> g_timeline{nullptr};
#endif


bool shape_ok_B(int32_t B) { return B >= 0 && B <= (1 << 24); }

int check_cfg(const switchsd_cfg *cfg) {
    if (!cfg)
        return SWITCHSD_EINVAL;
    if (cfg->n_ngram < 1 || cfg->n_ngram > SWITCHSD_MAX_NGRAM)
        return SWITCHSD_EINVAL;
    for (int j = 0; j < cfg->n_ngram; ++j) {
        const int n = cfg->ngram_lens[j];
        if (n < 1 || n > SWITCHSD_MAX_NGRAM_LEN)
            return SWITCHSD_EINVAL;
        if (j > 0 && n >= cfg->ngram_lens[j - 1])
            return SWITCHSD_EINVAL;
    }
    if (cfg->kappa < 1 || cfg->k < 0 || cfg->n_cand < 0 || cfg->n_cand > SWITCHSD_MAX_CAND)
        return SWITCHSD_EINVAL;
    return SWITCHSD_OK;
}

int32_t n_cand_of(int32_t n_cand) { return n_cand > 1 ? n_cand : 1; }

// Nodes of the longest copy draft: the anchor and W candidates of k tokens.
int64_t copy_nodes(const switchsd_cfg *cfg) {
    return 1 + (int64_t)n_cand_of(cfg->n_cand) * cfg->k;
}

void fill_cfg(StepParams &p, const switchsd_cfg *cfg) {
    p.n_ngram = cfg->n_ngram;
    for (int j = 0; j < SWITCHSD_MAX_NGRAM; ++j)
        p.lens[j] = j < cfg->n_ngram ? cfg->ngram_lens[j] : 0;
    p.nmax = cfg->ngram_lens[0];
    p.kappa = cfg->kappa;
    p.k = cfg->k;
    p.theta = cfg->theta;
    p.W = n_cand_of(cfg->n_cand);
}

int check_workspace(const void *ws, size_t bytes, int32_t B, int32_t R, int32_t Lmax,
                    int32_t W) {
    if (!ws || ((uintptr_t)ws & (kAlign - 1)))
        return SWITCHSD_EWORKSPACE;
    if (bytes < switchsd_workspace_bytes(B, R, Lmax, W))
        return SWITCHSD_EWORKSPACE;
    return SWITCHSD_OK;
}

int32_t key_stride_for(int32_t R) {
    return (int32_t)(((int64_t)R + kLineU64 - 1) / kLineU64 * kLineU64);
}

// Slots of a sequence's window table (copy labels): a power of two of at
// least 4 Lmax (the table is at most a quarter full, which keeps the probe
// walks short) and 64.
int64_t label_table_slots(int32_t Lmax) {
    int64_t t = 64;
    while (t < 4 * (int64_t)Lmax)
        t <<= 1;
    return t;
}

// Per-segment row maxima of the fused step (R <= 64 only): R * kMaxSegs
// keys per sequence on whole lines.
int32_t skey_stride_for(int32_t R) {
    if (R > 64)
        return 0;
    return (int32_t)(((int64_t)R * kMaxSegs + kLineU64 - 1) / kLineU64 * kLineU64);
}

// Per-tile match slots of a sequence whose context has 2..kMaxPollTiles scan
// tiles (8 per tile, on whole lines).
int32_t tslot_stride_for(int32_t Lmax) {
    const int64_t tiles = Lmax > 0 ? ((int64_t)Lmax + kScanTile - 1) / kScanTile : 0;
    if (tiles <= 1 || tiles > kMaxPollTiles)
        return 0;
    return (int32_t)((tiles * SWITCHSD_MAX_NGRAM + kLineU32 - 1) / kLineU32 * kLineU32);
}

int32_t rtk_stride_for(int32_t R) {
    return (int32_t)(((int64_t)R + kLineU32 - 1) / kLineU32 * kLineU32);
}

int scan_tiles_for(int32_t Lmax) { return (int)((Lmax + kScanTile - 1) / kScanTile); }

// int32 per sequence of the candidate lists: every scan tile keeps W ends per
// n-gram length; needed only with several candidates and several tiles.
int64_t cand_stride_for(int32_t Lmax, int32_t W) {
    const int64_t tiles = Lmax > 0 ? scan_tiles_for(Lmax) : 0;
    if (W <= 1 || tiles <= 1)
        return 0;
    return (tiles * SWITCHSD_MAX_NGRAM * W + kLineU32 - 1) / kLineU32 * kLineU32;
}

Workspace carve(void *ws, int32_t B, int32_t R, int32_t Lmax, int32_t W) {
    Workspace w;
    char *base = (char *)ws;
    const size_t line = (size_t)kLineU32 * 4;
    w.tk_front = (uint32_t *)base;
    w.tk_all = (uint32_t *)(base + (size_t)B * line);
    w.mslot = (int32_t *)(base + 2 * (size_t)B * line);
    w.keys = (unsigned long long *)(base + 3 * (size_t)B * line);
    w.key_stride = key_stride_for(R);
    w.qkeys = w.keys + (size_t)B * w.key_stride;
    w.rtk = (uint32_t *)(w.qkeys + (size_t)B * w.key_stride);
    w.rtk_stride = rtk_stride_for(R);
    w.skeys = (unsigned long long *)((char *)w.rtk + (size_t)B * w.rtk_stride * 4);
    w.skey_stride = skey_stride_for(R);
    w.tslot = (int32_t *)(w.skeys + (size_t)B * w.skey_stride);
    w.tslot_stride = tslot_stride_for(Lmax);
    w.cand = w.tslot + (size_t)B * w.tslot_stride;
    w.cand_stride = (int32_t)cand_stride_for(Lmax, W);
    return w;
}

// Compute units of the current device (cached per device).
int cu_count(int *out) {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return SWITCHSD_EHIP;
    if (dev >= 0 && dev < 64 && cache[dev] > 0) {
        *out = cache[dev];
        return SWITCHSD_OK;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
        return SWITCHSD_EHIP;
    if (dev >= 0 && dev < 64)
        cache[dev] = n;
    *out = n;
    return SWITCHSD_OK;
}

// Split each of `rows` logits rows into segments so that the argmax role has
// about two work-groups per compute unit, each segment at least one 16 KB
// chunk long and at most seg_cap segments per row.  Sets p.segs and
// p.seg_elems.
int set_segments(StepParams &p, int64_t rows, int32_t V, int64_t seg_cap = kMaxSegs) {
    int cus = 0;
    const int rc = cu_count(&cus);
    if (rc)
        return rc;
    const int64_t nvec = ((int64_t)V + 7) / 8;
    int64_t segs = (2 * (int64_t)cus + rows - 1) / rows;
    const int64_t max_segs = nvec / kChunkVecs > 1 ? nvec / kChunkVecs : 1;
    if (segs > max_segs)
        segs = max_segs;
    if (segs > seg_cap)
        segs = seg_cap;
    if (segs < 1)
        segs = 1;
    int64_t seg_elems = ((V + segs - 1) / segs + 7) / 8 * 8;
    segs = (V + seg_elems - 1) / seg_elems;
    p.segs = (int32_t)segs;
    p.seg_elems = (int32_t)seg_elems;
    return SWITCHSD_OK;
}

bool grid_ok(int64_t g) { return g >= 1 && g <= 0x7FFFFFFFll; }

int set_scan(StepParams &p, int32_t B, int32_t Lmax) {
    p.scan_tiles = scan_tiles_for(Lmax);
    const int64_t n = (int64_t)B * p.scan_tiles;
    if (n > 0x3FFFFFFFll)
        return SWITCHSD_ESHAPE;
    p.n_scan_wg = (int32_t)n;
    return SWITCHSD_OK;
}

}  // namespace

extern "C" {

size_t switchsd_workspace_bytes(int32_t B, int32_t R, int32_t Lmax, int32_t n_cand) {
    if (B < 0 || R < 0 || Lmax < 0 || n_cand < 0)
        return 0;
    // per sequence: three 256-byte lines (two tickets, the n-gram slots), the
    // row keys of the target's and of the draft's distribution, the row
    // tickets of the draw at T > 0, the per-segment row keys of the fused
    // step, the per-tile match slots and the candidate lists, each rounded up
    // to whole lines
    const int64_t W = n_cand > SWITCHSD_MAX_CAND ? SWITCHSD_MAX_CAND : n_cand_of(n_cand);
    return (size_t)B * ((size_t)kLineU32 * 4 * 3 + (size_t)key_stride_for(R) * 8 * 2 +
                        (size_t)rtk_stride_for(R) * 4 + (size_t)skey_stride_for(R) * 8 +
                        (size_t)tslot_stride_for(Lmax) * 4 +
                        (size_t)cand_stride_for(Lmax, (int32_t)W) * 4);
}

const char *switchsd_status_string(int status) {
    switch (status) {
    case SWITCHSD_OK:
        return "ok";
    case SWITCHSD_EINVAL:
        return "invalid argument (null pointer or bad configuration value)";
    case SWITCHSD_ESHAPE:
        return "sizes out of range or inconsistent";
    case SWITCHSD_EHIP:
        return "HIP runtime call or kernel launch failed";
    case SWITCHSD_EWORKSPACE:
        return "workspace null, not 256-byte aligned or too small";
    case SWITCHSD_ESCRATCH:
        return "the call needs more scratch than switchsd_step_noalloc holds "
               "(SWITCHSD_NOALLOC_SCRATCH_BYTES)";
    case SWITCHSD_EDEVICE:
        return "a bounded device-side wait gave up (results of that call are not valid; "
               "zero the workspace again)";
    default:
        return "unknown status";
    }
}

int switchsd_ngram_match(const int32_t *tokens, const int32_t *lengths, int32_t B, int32_t Lmax,
                         const switchsd_cfg *cfg, int32_t *match_n, int32_t *match_end,
                         int32_t *copy_len, int32_t *copy_tokens, void *workspace,
                         size_t workspace_bytes, hipStream_t stream) {
    int rc = check_cfg(cfg);
    if (rc)
        return rc;
    if (!shape_ok_B(B) || Lmax < 1)
        return SWITCHSD_ESHAPE;
    if (B == 0)
        return SWITCHSD_OK;
    if (!tokens || !lengths || !match_n || !match_end || !copy_len ||
        (cfg->k > 0 && !copy_tokens))
        return SWITCHSD_EINVAL;
    StepParams p;
    memset(&p, 0, sizeof p);
    fill_cfg(p, cfg);
    if ((rc = check_workspace(workspace, workspace_bytes, B, 0, Lmax, p.W)))
        return rc;
    p.tokens = tokens;
    p.lengths = lengths;
    p.B = B;
    p.Lmax = Lmax;
    p.R = 1;
    p.match_n = match_n;
    p.match_end = match_end;
    p.copy_len = copy_len;
    p.copy_tokens = copy_tokens;
    p.ws = carve(workspace, B, 0, Lmax, p.W);
    if ((rc = set_scan(p, B, Lmax)))
        return rc;
    p.n_front_wg = p.n_scan_wg;
    p.epi_front = EPI_MATCH;
    p.exp_front = (uint32_t)p.scan_tiles;
    return launch_step_kernel(p, p.n_front_wg, stream);
}

int switchsd_probe_score(const uint16_t *hidden, const float *w, float bias, int32_t B,
                         int32_t d, float *z, hipStream_t stream) {
    if (!shape_ok_B(B) || d < 0)
        return SWITCHSD_ESHAPE;
    if (B == 0)
        return SWITCHSD_OK;
    if (!z || (d > 0 && (!hidden || !w)))
        return SWITCHSD_EINVAL;
    StepParams p;
    memset(&p, 0, sizeof p);
    p.hidden = hidden;
    p.w = w;
    p.bias = bias;
    p.B = B;
    p.d = d;
    p.z = z;
    p.probe_on = 1;
    p.n_front_wg = B;
    return launch_step_kernel(p, B, stream);
}

int switchsd_select_draft(const int32_t *match_n, const int32_t *copy_len,
                          const int32_t *copy_tokens, const float *z, const int32_t *ntok,
                          const int32_t *npar, const int32_t *nn, int32_t B, int32_t R,
                          const switchsd_cfg *cfg, int32_t *use_copy, int32_t *dtok,
                          int32_t *dpar, int32_t *dn, hipStream_t stream) {
    int rc = check_cfg(cfg);
    if (rc)
        return rc;
    if (!shape_ok_B(B) || R < 1 || R > SWITCHSD_MAX_R || copy_nodes(cfg) > R)
        return SWITCHSD_ESHAPE;
    if (B == 0)
        return SWITCHSD_OK;
    if (!match_n || !copy_len || (cfg->k > 0 && !copy_tokens) || !z || !ntok || !nn ||
        !use_copy || !dtok || !dpar || !dn)
        return SWITCHSD_EINVAL;
    StepParams p;
    memset(&p, 0, sizeof p);
    fill_cfg(p, cfg);
    p.match_n_in = match_n;
    p.copy_len_in = copy_len;
    p.copy_tokens_in = copy_tokens;
    p.z_in = z;
    p.ntok = ntok;
    p.npar = npar;
    p.nn = nn;
    p.B = B;
    p.R = R;
    p.use_copy = use_copy;
    p.dtok = dtok;
    p.dpar = dpar;
    p.dn = dn;
    return launch_select_kernel(p, stream);
}

}  // extern "C"

namespace {

// Arguments of a verification at T > 0.
struct SampleArgs {
    float temperature;
    const uint64_t *uniforms;
    void *ws;
    size_t bytes;
    const uint16_t *qlogits;          // the draft's logits (speculative sampling with q) or null
    const uint64_t *accept_uniforms;  // [B, R] with qlogits
    const int32_t *spec_copy;         // the step's use_copy (copy drafts stay one-hot) or null
};

int64_t chunks_per_row(int32_t V) { return ((int64_t)V / 8 + kChunkVecs - 1) / kChunkVecs; }

size_t round_line(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

// The sample workspace: weight sums of the p rows and of the q rows per
// (chunk, wave), the residual sums of one row per sequence (128-bit per
// (chunk, wave)) and the test result of every row.
size_t csum_bytes(int32_t B, int32_t R, int32_t V) {
    return round_line((size_t)B * R * chunks_per_row(V) * kCsumPerChunk * 8);
}
size_t rcsum_bytes(int32_t B, int32_t V) {
    // per block of 64 vectors of one row per sequence: 4 u64
    return round_line((size_t)B * chunks_per_row(V) * (kChunkVecs / 64) * 32);
}

// The arguments of a draw at T > 0 other than its scratch.
int check_sample_args(const SampleArgs *sa, const uint16_t *logits, int32_t V) {
    if (!(sa->temperature > 0.0f) || !isfinite(sa->temperature) || !sa->uniforms)
        return SWITCHSD_EINVAL;
    if (V % 8 != 0 || ((uintptr_t)logits & 15))
        return SWITCHSD_EINVAL;
    if (sa->qlogits && (!sa->accept_uniforms || ((uintptr_t)sa->qlogits & 15)))
        return SWITCHSD_EINVAL;
    if (chunks_per_row(V) * (kThreads / 64) > kThreads)
        return SWITCHSD_ESHAPE;
    return SWITCHSD_OK;
}

int check_sample(const SampleArgs *sa, const uint16_t *logits, int32_t B, int32_t R, int32_t V) {
    const int rc = check_sample_args(sa, logits, V);
    if (rc)
        return rc;
    if (!sa->ws || ((uintptr_t)sa->ws & (kAlign - 1)) ||
        sa->bytes < switchsd_sample_workspace_bytes(B, R, V))
        return SWITCHSD_EWORKSPACE;
    return SWITCHSD_OK;
}

SampleArgs sample_args_of(const switchsd_step_args *a) {
    // speculative sampling with the neural draft's q (chains; copy drafts
    // stay one-hot)
    return SampleArgs{a->temperature,  a->uniforms,        a->sample_workspace,
                      a->sample_workspace_bytes, a->draft_logits, a->accept_uniforms,
                      a->use_copy};
}

// The sample workspace's regions and the draw's parameters in p.
void sample_carve(StepParams &p, const SampleArgs *sa) {
    p.uniforms = sa->uniforms;
    p.samp_c = (float)(1.4426950408889634 / (double)sa->temperature);
    p.cpr = (int32_t)chunks_per_row(p.V);
    char *sw = (char *)sa->ws;
    p.csum = (unsigned long long *)sw;
    p.qcsum = (unsigned long long *)(sw + csum_bytes(p.B, p.R, p.V));
    p.rcsum = (unsigned long long *)(sw + 2 * csum_bytes(p.B, p.R, p.V));
    p.rdec = (uint32_t *)(sw + 2 * csum_bytes(p.B, p.R, p.V) + rcsum_bytes(p.B, p.V));
    p.rz = (unsigned long long *)((char *)p.rdec + round_line((size_t)p.B * p.R * 4));
    p.qlogits = sa->qlogits;
    p.accept_uniforms = sa->accept_uniforms;
    p.spec_copy = sa->spec_copy;
}

// The polled draw: one-hot drafts (no q) of at most 64 rows, and at most one
// waiting work-group per compute unit on average (the first segment's of each
// of the B * R rows, first in the sum launch's grid), so that they cannot hold
// every slot the other work-groups need; those wait for nothing.
bool draw_polled(const StepParams &p, const SampleArgs *sa, int cus) {
    return !sa->qlogits && p.R <= 64 && p.ws.skey_stride > 0 && (int64_t)p.B * p.R <= cus;
}

// The row maxima launch before a draw: with the polled draw, it also zeroes
// the sum slots (csum_clear), so the sample workspace needs no initialization.
int prepare_draw(StepParams &p, const SampleArgs *sa) {
    int cus = 0;
    const int rc = cu_count(&cus);
    if (rc)
        return rc;
    sample_carve(p, sa);
    p.csum_clear = draw_polled(p, sa, cus) ? 1 : 0;
    return SWITCHSD_OK;
}

// After the row maxima are in the row keys: the weight-sum launch, which also
// draws each row's token and runs the accept epilogue.  With the draft's q:
// first the q row maxima, then the sums of the p and the q rows (the last
// work-group of a row with a drafted child takes its accept test), then the
// residual launch, which draws the emitted token where the chain ends and
// writes the outputs.  `p` carries the rows, the draft, the outputs and the
// carved workspace.
int sample_finish(StepParams p, const SampleArgs *sa, bool speculate, hipStream_t stream) {
    int cus = 0;
    int rc = cu_count(&cus);
    if (rc)
        return rc;
    const bool q = sa->qlogits != nullptr;
    p.tl = nullptr;  // phase stamps (timeline build) cover the step kernel's grid only
    // long drafts: the sums stream the drafted rows' chunks over a fixed grid
    const bool stream_sums = p.R > 64 && p.B <= kListMaxB && !q;
    sample_carve(p, sa);
    // the polled draw when the maxima launch cleared its slots
    const bool polled = p.csum_clear && !stream_sums;
    p.csum_clear = 0;
    const int64_t rows = (int64_t)p.B * p.R;
    if (q && !p.qmax) {
        // the q row maxima: the argmax role alone, over the rows with a
        // drafted child of the sequences verified with q
        StepParams pq = p;
        pq.logits = sa->qlogits;
        pq.ws.keys = p.ws.qkeys;
        pq.n_front_wg = pq.n_scan_wg = pq.n_poll_wg = 0;
        pq.poll_accept = 0;
        pq.csum_clear = 0;
        pq.qmax = 0;
        pq.probe_on = pq.scan_probe = 0;
        pq.epi_front = EPI_NONE;
        pq.epi_accept = 0;
        pq.list_mode = 0;
        pq.speculate = 0;
        pq.commit = 0;
        pq.rows_mode = ROWS_Q;
        if ((rc = set_segments(pq, rows, p.V)))
            return rc;
        const int64_t g = rows * pq.segs;
        if (!grid_ok(g))
            return SWITCHSD_ESHAPE;
        if ((rc = launch_step_kernel(pq, g, stream)))
            return rc;
    }
    // about six sum work-groups per CU, as many as stay resident (with q,
    // three for the p rows and three for the q rows).  Measured on C2 at
    // T = 0.7 (16 chunks per row): 2, 3, 4, 6, 8 and 16 per CU gave 42.2,
    // 39.1, 39.6, 38.6, 40.2 and 42.8 us per step; with q, six per CU per
    // tensor (two batches) 80.2 us against 77.4 us for three.
    int64_t segs = ((q ? 3 : 6) * (int64_t)cus + rows - 1) / rows;
    if (segs > p.cpr)
        segs = p.cpr;
    if (segs < 1)
        segs = 1;
    p.seg_chunks = (int32_t)((p.cpr + segs - 1) / segs);
    p.segs = (int32_t)((p.cpr + p.seg_chunks - 1) / p.seg_chunks);
    p.speculate = speculate ? 1 : 0;
    p.list_mode = stream_sums ? 1 : 0;
    p.draw_poll = polled ? 1 : 0;
    const int64_t grid = stream_sums ? 4 * (int64_t)cus : rows * p.segs * (q ? 2 : 1);
    if (!grid_ok(grid) || !grid_ok(rows))
        return SWITCHSD_ESHAPE;
    // polled: the first work-group of row r draws its token and row 0's runs
    // the accept epilogue; else the last work-group of each drafted row draws its token
    // (or takes its accept test), and the last drafted row of a sequence runs
    // the accept epilogue (sequences verified with q: the residual launch does)
    if ((rc = launch_sample_sums_kernel(p, grid, stream)) || !q)
        return rc;
    // residual: one work-group per 512 vectors (8 KB) of the rejected row,
    // two blocks of 64 vectors per wave, covering every block of every chunk
    // (the draw sums 16 block entries per chunk; blocks past the row's end
    // write zero)
    p.rsegs = p.cpr * (kChunkVecs / kThreads) / 2;
    const int64_t rgrid = (int64_t)p.B * p.rsegs;
    if (!grid_ok(rgrid))
        return SWITCHSD_ESHAPE;
    return launch_spec_residual_kernel(p, rgrid, stream);
}

// Verify launch shared by the entry points and the split step.  `speculate`:
// most rows of the drafts are expected to be read (chains), so a row's first
// chunk is requested before its need is known.  With `sa`, the launch only
// leaves the row maxima and the draw at T > 0 follows.
int verify_launch(const uint16_t *logits, int32_t B, int32_t R, int32_t V, const int32_t *dtok,
                  const int32_t *dpar, const int32_t *dn, int32_t *accept_len,
                  int32_t *accept_node, int32_t *bonus, int32_t *out_tokens, int32_t *amax,
                  void *workspace, size_t workspace_bytes, bool speculate,
                  const SampleArgs *sa, const StepParams *loop, hipStream_t stream) {
    if (!shape_ok_B(B) || R < 1 || R > SWITCHSD_MAX_R || V < 1)
        return SWITCHSD_ESHAPE;
    if (B == 0)
        return SWITCHSD_OK;
    if (!logits || ((uintptr_t)logits & 1) || !dtok || !dn || !accept_len || !accept_node ||
        !bonus || !out_tokens)
        return SWITCHSD_EINVAL;
    int rc = check_workspace(workspace, workspace_bytes, B, R, 0, 0);
    if (rc)
        return rc;
    if (sa && (rc = check_sample(sa, logits, B, R, V)))
        return rc;
    StepParams p;
    memset(&p, 0, sizeof p);
    p.W = 1;
    int64_t grid = 0;
    if (R > 64 && B <= kListMaxB && V % 8 == 0 && ((uintptr_t)logits & 15) == 0 &&
        (int64_t)B * R * ((V / 8 + kChunkVecs - 1) / kChunkVecs) < 0x7FFFFFFFll) {
        // long drafts use few of their rows: a fixed grid streams the chunks
        // of the drafted rows, split evenly
        int cus = 0;
        if ((rc = cu_count(&cus)))
            return rc;
        p.segs = (V / 8 + kChunkVecs - 1) / kChunkVecs;  // chunks per row
        p.list_mode = 1;
        grid = 4 * (int64_t)cus;
    } else {
        // At T = 0 with R <= 64 and B no larger than the CU count, one
        // work-group per sequence (first in the grid) holds the draft and
        // polls the segment results (as the fused step's front does); the
        // other work-groups wait for nothing.
        int cus = 0;
        if ((rc = cu_count(&cus)))
            return rc;
        const bool poll = !sa && R <= 64 && B <= cus;
        const int64_t cap = poll && kMaxPollSlots / R < kMaxSegs ? kMaxPollSlots / R : kMaxSegs;
        if ((rc = set_segments(p, (int64_t)B * R, V, cap)))
            return rc;
        if (poll) {
            p.poll_accept = 1;
            p.n_poll_wg = B;
        }
        // with the draft's q the same launch also takes the q row maxima
        p.qmax = sa && sa->qlogits && p.W == 1 ? 1 : 0;
        grid = p.n_poll_wg + (int64_t)B * R * p.segs * (1 + p.qmax);
        if (!grid_ok(grid))
            return SWITCHSD_ESHAPE;
    }
    p.logits = logits;
    p.B = B;
    p.R = R;
    p.V = V;
    p.dtok = const_cast<int32_t *>(dtok);
    p.dpar = const_cast<int32_t *>(dpar);
    p.dn = const_cast<int32_t *>(dn);
    p.accept_len = accept_len;
    p.accept_node = accept_node;
    p.bonus = bonus;
    p.out_tokens = out_tokens;
    p.amax = amax;
    p.ws = carve(workspace, B, R, 0, 0);
    p.rows_mode = p.list_mode ? ROWS_LISTED : ROWS_DRAFT;
    p.speculate = speculate && !p.list_mode ? 1 : 0;
    p.epi_accept = sa ? 0 : 1;
    if (loop && loop->commit) {  // the decode loop's commit rides on the accept epilogue
        p.commit = 1;
        p.ctok = loop->ctok;
        p.clen = loop->clen;
        p.draft_pos = loop->draft_pos;
        p.lag = loop->lag;
        p.Lmax = loop->Lmax;
        p.use_copy = loop->use_copy;
    }
    p.exp_all = (uint32_t)(R * p.segs);
    p.spin_cap = 1 << 22;  // the bound of each poll (see switchsd_workspace_status)
    if (sa && (rc = prepare_draw(p, sa)))
        return rc;
    if ((rc = launch_step_kernel(p, grid, stream)) || !sa)
        return rc;
    return sample_finish(p, sa, speculate, stream);
}

}  // namespace

namespace switchsd {

// Every check of switchsd_step's arguments except its two workspaces.
int check_step_args(const switchsd_step_args *a) {
    if (!a)
        return SWITCHSD_EINVAL;
    int rc = check_cfg(&a->cfg);
    if (rc)
        return rc;
    const int32_t B = a->B, R = a->R, V = a->V;
    if (!shape_ok_B(B) || a->Lmax < 1 || a->d < 0 || R < 1 || R > SWITCHSD_MAX_R || V < 1 ||
        copy_nodes(&a->cfg) > R)
        return SWITCHSD_ESHAPE;
    if (a->mode < SWITCHSD_MODE_AUTO || a->mode > SWITCHSD_MODE_SPLIT)
        return SWITCHSD_EINVAL;
    if (B == 0)
        return SWITCHSD_OK;
    if (!a->tokens || !a->lengths || (a->d > 0 && (!a->hidden || !a->w)) || !a->ntok ||
        !a->nn || !a->logits || ((uintptr_t)a->logits & 1) || !a->match_n || !a->match_end ||
        !a->copy_len || (a->cfg.k > 0 && !a->copy_tokens) || !a->z || !a->use_copy ||
        !a->dtok || !a->dpar || !a->dn || !a->accept_len || !a->accept_node || !a->bonus ||
        !a->out_tokens || (a->commit && (!a->draft_pos || !a->lag)))
        return SWITCHSD_EINVAL;
    const bool sampled = a->temperature != 0.0f;
    if (a->draft_logits && (!sampled || a->npar))
        return SWITCHSD_EINVAL;
    const SampleArgs sa = sample_args_of(a);
    if (sampled && (rc = check_sample_args(&sa, a->logits, V)))
        return rc;
    return SWITCHSD_OK;
}

}  // namespace switchsd

extern "C" {

int switchsd_verify_accept(const uint16_t *logits, int32_t B, int32_t R, int32_t V,
                           const int32_t *dtok, const int32_t *dpar, const int32_t *dn,
                           int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                           int32_t *out_tokens, int32_t *amax, void *workspace,
                           size_t workspace_bytes, hipStream_t stream) {
    // chains and short drafts usually use every row
    const bool speculate = dpar == nullptr || R <= 16;
    return verify_launch(logits, B, R, V, dtok, dpar, dn, accept_len, accept_node, bonus,
                         out_tokens, amax, workspace, workspace_bytes, speculate, nullptr,
                         nullptr, stream);
}

int switchsd_verify_sample(const uint16_t *logits, int32_t B, int32_t R, int32_t V,
                           float temperature, const uint64_t *uniforms,
                           const uint16_t *draft_logits, const uint64_t *accept_uniforms,
                           const int32_t *dtok, const int32_t *dpar, const int32_t *dn,
                           int32_t *accept_len, int32_t *accept_node, int32_t *bonus,
                           int32_t *out_tokens, int32_t *amax, void *workspace,
                           size_t workspace_bytes, void *sample_workspace,
                           size_t sample_workspace_bytes, hipStream_t stream) {
    const SampleArgs sa = {temperature,  uniforms,        sample_workspace, sample_workspace_bytes,
                           draft_logits, accept_uniforms, nullptr};
    if (draft_logits && dpar)  // speculative sampling with q: chains only
        return SWITCHSD_EINVAL;
    const bool speculate = dpar == nullptr || R <= 16;
    return verify_launch(logits, B, R, V, dtok, dpar, dn, accept_len, accept_node, bonus,
                         out_tokens, amax, workspace, workspace_bytes, speculate, &sa, nullptr,
                         stream);
}

size_t switchsd_sample_workspace_bytes(int32_t B, int32_t R, int32_t V) {
    if (B < 0 || R < 0 || V < 0)
        return 0;
    return 2 * csum_bytes(B, R, V) + rcsum_bytes(B, V) + round_line((size_t)B * R * 4) +
           round_line((size_t)B * R * 16);
}

int switchsd_step(const switchsd_step_args *a, void *workspace, size_t workspace_bytes,
                  hipStream_t stream) {
    int rc = check_step_args(a);
    if (rc || a->B == 0)
        return rc;
    const int32_t B = a->B, R = a->R, V = a->V;
    StepParams p;
    memset(&p, 0, sizeof p);
    fill_cfg(p, &a->cfg);
    if ((rc = check_workspace(workspace, workspace_bytes, B, R, a->Lmax, p.W)))
        return rc;
    p.withhold_flag = g_withhold_probe_flag.load() ? 1 : 0;
    p.withhold_seg = g_withhold_segment.load() ? 1 : 0;
    p.spin_cap = p.withhold_flag || p.withhold_seg ? 256 : (1 << 22);
#ifdef SWITCHSD_TIMELINE
    p.tl = g_timeline.load();
#endif
    const bool sampled = a->temperature != 0.0f;
    const SampleArgs sa = sample_args_of(a);
    if (sampled && (rc = check_sample(&sa, a->logits, B, R, V)))
        return rc;
    p.tokens = a->tokens;
    p.lengths = a->lengths;
    p.hidden = a->hidden;
    p.w = a->w;
    p.ntok = a->ntok;
    p.npar = a->npar;
    p.nn = a->nn;
    p.logits = a->logits;
    p.B = B;
    p.Lmax = a->Lmax;
    p.d = a->d;
    p.R = R;
    p.V = V;
    p.bias = a->bias;
    p.match_n = a->match_n;
    p.match_end = a->match_end;
    p.copy_len = a->copy_len;
    p.copy_tokens = a->copy_tokens;
    p.z = a->z;
    p.use_copy = a->use_copy;
    p.dtok = a->dtok;
    p.dpar = a->dpar;
    p.dn = a->dn;
    p.amax = a->amax;
    p.accept_len = a->accept_len;
    p.accept_node = a->accept_node;
    p.bonus = a->bonus;
    p.out_tokens = a->out_tokens;
    if (a->commit) {
        p.commit = 1;
        p.ctok = const_cast<int32_t *>(a->tokens);
        p.clen = const_cast<int32_t *>(a->lengths);
        p.draft_pos = a->draft_pos;
        p.lag = a->lag;
    }
    p.ws = carve(workspace, B, R, a->Lmax, p.W);
    if ((rc = set_scan(p, B, a->Lmax)))
        return rc;
    // one tile: it computes the probe too; several: the probe has a work-group
    // of its own (first in the grid) and no tile carries it
    if (p.scan_tiles > 1) {
        p.probe_on = 1;
        p.n_front_wg = p.n_scan_wg + B;
    } else {
        p.scan_probe = 1;
        p.n_front_wg = p.n_scan_wg;
    }
    p.epi_front = EPI_SELECT;
    p.exp_front = (uint32_t)p.scan_tiles;
    // One waiting work-group per sequence (the last scan tile) and at most one
    // per compute unit; every other work-group of the grid runs to completion
    // without waiting.
    int cus = 0;
    if ((rc = cu_count(&cus)))
        return rc;
    p.poll_front = p.ws.tslot_stride > 0 && B <= cus ? 1 : 0;

    const int64_t cn = copy_nodes(&a->cfg);
    int mode = a->mode;
    if (mode == SWITCHSD_MODE_AUTO)  // short drafts that may use every row: one launch
        mode = cn >= R && R <= 64 ? SWITCHSD_MODE_FUSED : SWITCHSD_MODE_SPLIT;
    if (mode == SWITCHSD_MODE_FUSED) {
        // the accept epilogue polls at most kMaxPollSlots segment results
        const int64_t cap = kMaxPollSlots / R < kMaxSegs ? kMaxPollSlots / R : kMaxSegs;
        if ((rc = set_segments(p, (int64_t)B * R, V, cap < 1 ? 1 : cap)))
            return rc;
        // with the draft's q the same launch also takes the q row maxima
        // (before the draft is chosen: the neural draft's rows)
        p.qmax = sampled && sa.qlogits && p.W == 1 ? 1 : 0;
        const int64_t grid = p.n_front_wg + (int64_t)B * R * p.segs * (1 + p.qmax);
        if (!grid_ok(grid))
            return SWITCHSD_ESHAPE;
        p.rows_mode = cn >= R ? ROWS_ALL : ROWS_NEURAL_OR_COPY;
        p.epi_accept = sampled ? 0 : 1;
        p.exp_all = p.exp_front + (uint32_t)(R * p.segs);
        // The accept epilogue polls the segment slots from the front's
        // work-group when at most one such waiting work-group per compute
        // unit exists: every other work-group of the grid runs to completion
        // without waiting, so the waiting ones cannot hold every slot the
        // argmax work-groups need.
        p.poll_accept = !sampled && p.W == 1 && R <= 64 &&
                                (int64_t)R * p.segs <= kMaxPollSlots && B <= cus
                            ? 1
                            : 0;
        if (sampled && (rc = prepare_draw(p, &sa)))
            return rc;
        if ((rc = launch_step_kernel(p, grid, stream)) || !sampled)
            return rc;
        return sample_finish(p, &sa, true, stream);
    }
    // SPLIT: front (scan + probe + select), then verify over the chosen rows
    if ((rc = launch_step_kernel(p, p.n_front_wg, stream)))
        return rc;
    // rows past a draft are skipped; only short drafts request a row's first
    // chunk before its need is known
    return verify_launch(a->logits, B, R, V, a->dtok, a->dpar, a->dn, a->accept_len,
                         a->accept_node, a->bonus, a->out_tokens, a->amax, workspace,
                         workspace_bytes, R <= 16, sampled ? &sa : nullptr, &p, stream);
}

size_t switchsd_label_workspace_bytes(int32_t B, int32_t Lmax) {
    if (B < 0 || Lmax < 0 || Lmax > (1 << 28))
        return 0;
    // a table of the distinct windows per sequence
    return (size_t)((int64_t)B * label_table_slots(Lmax) * 4);
}

int switchsd_copy_labels(const int32_t *tokens, const int32_t *lengths, int32_t B, int32_t Lmax,
                         int32_t n, uint8_t *labels, void *workspace, size_t workspace_bytes,
                         hipStream_t stream) {
    if (!shape_ok_B(B) || Lmax < 1 || Lmax > (1 << 28) ||
        (int64_t)B * label_table_slots(Lmax) * 4 > (1ll << 40))
        return SWITCHSD_ESHAPE;
    if (n < 1 || n > 64)
        return SWITCHSD_EINVAL;
    if (B == 0)
        return SWITCHSD_OK;
    if (!tokens || !lengths || !labels)
        return SWITCHSD_EINVAL;
    if (!workspace || ((uintptr_t)workspace & (kAlign - 1)) ||
        workspace_bytes < switchsd_label_workspace_bytes(B, Lmax))
        return SWITCHSD_EWORKSPACE;
    StepParams p;
    memset(&p, 0, sizeof p);
    p.tokens = tokens;
    p.lengths = lengths;
    p.B = B;
    p.Lmax = Lmax;
    const int64_t grid = (int64_t)B * ((Lmax + kThreads - 1) / kThreads);
    if (!grid_ok(grid))
        return SWITCHSD_ESHAPE;
    return launch_label_kernels(p, n, labels, (int32_t)label_table_slots(Lmax), workspace,
                                stream);
}

int switchsd_commit(int32_t *tokens, int32_t *lengths, int32_t B, int32_t Lmax,
                    const int32_t *out_tokens, int32_t R, const int32_t *accept_len,
                    const int32_t *use_copy, int32_t *draft_pos, int32_t *lag,
                    hipStream_t stream) {
    if (!shape_ok_B(B) || Lmax < 1 || R < 1 || R > SWITCHSD_MAX_R)
        return SWITCHSD_ESHAPE;
    if (B == 0)
        return SWITCHSD_OK;
    if (!tokens || !lengths || !out_tokens || !accept_len || !use_copy || !draft_pos || !lag)
        return SWITCHSD_EINVAL;
    StepParams p;
    memset(&p, 0, sizeof p);
    p.B = B;
    p.R = R;
    p.Lmax = Lmax;
    p.ctok = tokens;
    p.clen = lengths;
    p.out_tokens = const_cast<int32_t *>(out_tokens);
    p.accept_len = const_cast<int32_t *>(accept_len);
    p.use_copy = const_cast<int32_t *>(use_copy);
    p.draft_pos = draft_pos;
    p.lag = lag;
    return launch_commit_kernel(p, stream);
}

int switchsd_workspace_status(void *workspace, size_t workspace_bytes, int32_t B,
                              int32_t *status, hipStream_t stream) {
    if (!shape_ok_B(B))
        return SWITCHSD_ESHAPE;
    if (!status)
        return SWITCHSD_EINVAL;
    if (!workspace || ((uintptr_t)workspace & (kAlign - 1)) ||
        workspace_bytes < switchsd_workspace_bytes(B, 0, 0, 0))
        return SWITCHSD_EWORKSPACE;
    return launch_status_kernel(carve(workspace, B, 0, 0, 0).mslot, B, status, stream);
}

void switchsd_test_withhold_probe_flag(int32_t on) { g_withhold_probe_flag.store(on ? 1 : 0); }

void switchsd_test_withhold_segment(int32_t on) { g_withhold_segment.store(on ? 1 : 0); }

#ifdef SWITCHSD_TIMELINE
// Timeline build only (not part of the product library's interface): phase
// stamps of the following switchsd_step launches go to `buf` (device, 8 u64
// per work-group of the largest launch); NULL stops recording.
void switchsd_timeline_buffer(unsigned long long *buf) { g_timeline.store(buf); }
#endif

int switchsd_tree_mask(const int32_t *dpar, const int32_t *dn, int32_t B, int32_t R,
                       uint32_t *mask, hipStream_t stream) {
    if (!shape_ok_B(B) || R < 1 || R > SWITCHSD_MAX_R)
        return SWITCHSD_ESHAPE;
    if (B == 0)
        return SWITCHSD_OK;
    if (!dn || !mask)
        return SWITCHSD_EINVAL;
    const int64_t per = ((int64_t)R * ((R + 31) / 32) + kThreads - 1) / kThreads;
    if (!grid_ok((int64_t)B * per))
        return SWITCHSD_ESHAPE;
    return launch_tree_mask_kernel(dpar, dn, B, R, mask, stream);
}

}  // extern "C"
