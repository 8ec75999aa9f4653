// switchsd_internal.h -- parameters shared by the host API and the kernels.
// Not part of the public interface (see include/switchsd.h).
#pragma once

#include <stdint.h>

#include "switchsd.h"

namespace switchsd {

// Work-group shape of every kernel of the step: 256 lanes = 4 wave64s.
constexpr int kThreads = 256;
// 16-byte logits vectors per lane in one chunk of the argmax stream.
constexpr int kUnroll = 4;
// 16-byte vectors in one chunk (16 KB); two chunks are in flight per work-group.
constexpr int kChunkVecs = kThreads * kUnroll;
// Context end positions covered by one scan work-group.
constexpr int kScanTile = 1024;
// Weight sums per 16 KB chunk of the draw at T > 0: one per wave (each wave
// reads 256 contiguous vectors of the chunk).
constexpr int kCsumPerChunk = kThreads / 64;
// Per-sequence workspace slots live on their own 256-byte lines: atomics to
// one line serialize, and every work-group of a sequence arrives at its line.
constexpr int kLineU32 = 64;
constexpr int kLineU64 = 32;
// Copy candidates per sequence, at most.
constexpr int kMaxCand = SWITCHSD_MAX_CAND;
// Argmax segments per logits row, at most (the fused step's per-segment
// result slots hold R * kMaxSegs keys per sequence).
constexpr int kMaxSegs = 16;
// Workspace slots one poll of wave 0 covers, at most (8 per lane).
constexpr int kMaxPollSlots = 512;
// Scan tiles per sequence, at most, for which the last tile polls per-tile
// match slots instead of an arrival (the other tiles' 8 slots each).
constexpr int kMaxPollTiles = kMaxPollSlots / 8;

enum : int32_t { EPI_NONE = 0, EPI_MATCH = 1, EPI_SELECT = 2 };
enum : int32_t {
    ROWS_ALL = 0,
    ROWS_NEURAL_OR_COPY = 1,
    ROWS_DRAFT = 2,
    ROWS_LISTED = 3,
    ROWS_Q = 4  // the draft's rows r < dn - 1 of sequences verified with q
};
// Sequences a work-list verify launch handles (its item prefix sums live in
// four registers per lane).
constexpr int kListMaxB = 256;

struct Workspace {
    uint32_t *tk_front;        // [B] x 256 B: arrivals of the scan/probe work-groups
    uint32_t *tk_all;          // [B] x 256 B: arrivals of every work-group of a sequence
    int32_t *mslot;            // [B] x 256 B: most recent end + 1 per n-gram length
    unsigned long long *keys;  // [B] x key_stride: packed (value key, ~index) row maxima
    int32_t key_stride;        // u64 per sequence (R rounded up to a 256-byte line)
    uint32_t *rtk;             // [B] x rtk_stride: arrivals of the sum work-groups per row
                               // (draw at T > 0)
    int32_t rtk_stride;        // u32 per sequence (R rounded up to a 256-byte line)
    int32_t *cand;             // [B] x cand_stride: per scan tile and n-gram length, the
                               // tile's W most recent ends + 1 (0: none); W > 1 and
                               // more than one tile only
    int32_t cand_stride;       // int32 per sequence (whole 256-byte lines)
    unsigned long long *qkeys; // [B] x key_stride: row maxima of the draft's distribution q
                               // (between keys and rtk)
    unsigned long long *skeys; // [B] x skey_stride: the fused step's per-segment row maxima,
                               // segment s of row r at s * R + r (0: not yet written,
                               // 1: the segment has no candidate); between rtk and cand
    int32_t skey_stride;       // u64 per sequence (R * kMaxSegs on whole lines; 0 if R > 64)
    int32_t *tslot;            // [B] x tslot_stride: per scan tile t and n-gram length j at
                               // t * 8 + j, the tile's most recent end + 2 (1: none, 0: not
                               // yet written); between skeys and cand
    int32_t tslot_stride;      // int32 per sequence (tiles * 8 on whole lines; 0 unless
                               // 1 < tiles <= kMaxPollTiles)
};

struct StepParams {
    // inputs
    const int32_t *tokens;
    const int32_t *lengths;
    const uint16_t *hidden;
    const float *w;
    const int32_t *ntok;
    const int32_t *npar;
    const int32_t *nn;
    const uint16_t *logits;
    const int32_t *copy_tokens_in;  // select stage only
    const int32_t *match_n_in;      // select stage only
    const int32_t *copy_len_in;     // select stage only
    const float *z_in;              // select stage only
    int32_t B, Lmax, d, R, V;
    float bias;
    // configuration
    int32_t n_ngram;
    int32_t lens[SWITCHSD_MAX_NGRAM];
    int32_t nmax;
    int32_t kappa;
    int32_t k;
    float theta;
    int32_t W;  // copy candidates (>= 1)
    // outputs
    int32_t *match_n, *match_end, *copy_len, *copy_tokens;
    float *z;
    int32_t *use_copy, *dtok, *dpar, *dn;
    int32_t *amax;
    int32_t *accept_len, *accept_node, *bonus, *out_tokens;
    Workspace ws;
    // grid layout: [probe][scan tiles][argmax row segments, segment-major]
    int32_t scan_tiles;  // per sequence (0: no scan role)
    int32_t probe_on;    // 1: one probe work-group per sequence, first in the grid
    int32_t scan_probe;  // 1: scan tile 0 of each sequence also computes the probe
    int32_t segs;        // argmax work-groups per row (0: no argmax role)
    int32_t seg_elems;   // logits elements per row segment (multiple of 8)
    int32_t n_scan_wg;   // B * scan_tiles
    int32_t n_front_wg;  // n_scan_wg + B * probe_on
    int32_t rows_mode;
    int32_t speculate;   // 1: issue a row's first chunk before reading whether it is needed
    int32_t epi_front;
    int32_t epi_accept;
    int32_t poll_accept; // 1 (R <= 64, T = 0): each argmax work-group stores its result in
                         // its own slot, and the work-group holding the sequence's draft
                         // (the front's chooser in the fused step, a poller work-group
                         // in the verify launch) polls the slots and runs the accept
                         // epilogue (no arrivals at tk_all)
    int32_t n_poll_wg;   // verify launch with poll_accept: one waiting work-group per
                         // sequence, first in the grid, runs its accept epilogue
    int32_t poll_front;  // 1 (the step, 1 < scan_tiles <= kMaxPollTiles): each scan tile
                         // stores its match slots in its own line (with several candidates
                         // after its completed candidate lists) and the last tile polls
                         // them (no arrivals at tk_front)
    int32_t list_mode;   // 1: verify only, a fixed grid streaming the chunks of the drafted
                         // rows r < dn[b] (segs = chunks per row)
    // decode loop: the accept epilogue appends to the context (read-write)
    int32_t commit;
    int32_t *ctok;       // [B, Lmax] the context, written at positions >= its length
    int32_t *clen;       // [B] its length
    int32_t *draft_pos;  // [B] draft-model cache position (in/out)
    int32_t *lag;        // [B] tokens the next neural drafting pass must consume first
    // draws at T > 0 (the weight-sum launch)
    const uint64_t *uniforms;  // [B, R]
    float samp_c;              // log2(e) / T
    unsigned long long *csum;  // [B, R, cpr, waves] integer weight sums per chunk and wave
    int32_t cpr;               // 16 KB chunks per row
    int32_t seg_chunks;        // chunks per work-group of the sum launch
    int32_t draw_poll;         // 1: the polled draw (no q, R <= 64): sums stored + 1, the
                               // work-group of each row's first segment draws the row's token
                               // and row 0's runs the accept epilogue (no arrivals)
    int32_t csum_clear;        // the row maxima launch before a polled draw: each argmax
                               // work-group zeroes its share of its row's sum slots
    int32_t qmax;              // 1: the row maxima launch also takes the draft's q rows, its
                               // last B * R * segs work-groups (q keys); else a launch of
                               // their own follows
    // speculative sampling with the draft's own distribution q (chains, T > 0)
    const uint16_t *qlogits;          // [B, R, V] the draft's logits, or null (one-hot drafts)
    const uint64_t *accept_uniforms;  // [B, R] uniforms of the accept tests
    const int32_t *spec_copy;         // [B] use_copy of the step (copy drafts stay one-hot)
                                      // or null (every sequence uses q)
    unsigned long long *qcsum;        // [B, R, cpr, waves] integer weight sums of the q rows
    unsigned long long *rcsum;        // [B, cpr * 16, 4] per block of 64 vectors of the
                                      // rejected row: residual sum (lo, hi), P sum, unused
    uint32_t *rdec;                   // [B, R] test of row r: 1 accepted, 2 rejected
    unsigned long long *rz;           // [B, R, 2] Zp, Zq of each tested row
    int32_t rsegs;                    // residual work-groups per sequence (8 KB each)
    // bounded waits: spin limit of the front's wait for the probe flag and of
    // its poll of the segment slots; with withhold_flag (a test knob) the
    // probe never sets its flag
    int32_t spin_cap;
    int32_t withhold_flag;
    int32_t withhold_seg;  // test knob: sequence 0's row 0 segment 0 (of the argmax, and of the
                           // weight sums in a polled draw) and its scan tile 0 never store
                           // their slots
    unsigned long long *tl;  // timeline build only: per work-group phase stamps
    uint32_t exp_front;  // arrivals per sequence at tk_front
    uint32_t exp_all;    // arrivals per sequence at tk_all
};

// Every check of switchsd_step's arguments except its two workspaces
// (switchsd_step and switchsd_step_noalloc run it before anything else).
int check_step_args(const switchsd_step_args *a);

int launch_step_kernel(const StepParams &p, int64_t grid, hipStream_t stream);
int launch_select_kernel(const StepParams &p, hipStream_t stream);
int launch_commit_kernel(const StepParams &p, hipStream_t stream);
int launch_label_kernels(const StepParams &p, int32_t n, uint8_t *labels, int32_t tsize,
                         void *table, hipStream_t stream);
int launch_sample_sums_kernel(const StepParams &p, int64_t grid, hipStream_t stream);
int launch_spec_residual_kernel(const StepParams &p, int64_t grid, hipStream_t stream);
int launch_status_kernel(int32_t *mslot, int32_t B, int32_t *out, hipStream_t stream);
int launch_tree_mask_kernel(const int32_t *dpar, const int32_t *dn, int32_t B, int32_t R,
                            uint32_t *mask, hipStream_t stream);

}  // namespace switchsd
