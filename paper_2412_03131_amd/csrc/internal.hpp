// internal.hpp -- argument blocks and launchers shared by the API and kernels.
#pragma once

#include "common.hpp"

namespace dkv {

struct TState {        // per-table scratch of one append call
    int32_t cnt[2];    // kept new tokens per section
    int32_t lold[2];   // section lengths before the call
    int32_t pold[2];   // pages held before the call
    int32_t ring_off;  // first ring index of this table's new pages, from head_old
    int32_t n;         // new tokens of the table's sequence
};

struct LayoutArgs {
    int p_max;
    int T[2];
    int kb[2], vb[2];  // key and value bits per section
    int tsh;           // log2 of the tokens per page: high section in bits 0-7, low in 8-15
    long long page_bytes;
    int off_kcode[2], off_kmeta[2], off_vcode[2], off_vmeta[2], off_score[2], off_pos[2];
};

struct AppendArgs : LayoutArgs {
    uint8_t* pool;
    long long num_pages;
    int32_t* page_table;
    int32_t* pages;
    int32_t* len;
    int32_t* seq_len;
    int32_t* ring;
    int64_t* ring_ptr;
    uint32_t* status;
    int B, Hkv;
    long long total_new;
    int max_new;
    const int32_t* new_len;
    const uint16_t* k;
    const uint16_t* v;
    const float* score;
    const int32_t* quota;
    float alpha_h, alpha_l;
    int window;
    CallFlags* flags;
    TState* tstate;
    int32_t* sold;
    int32_t* row_off;
    int32_t* ord;
    long long* tplan;    // [tables] exclusive prefix (new pages | jobs << 32), planned path
    int32_t* job_table;  // [job_cap] table of each page job, planned path
    int job_cap;
};

// Above this many tables an append plans once in its own launch instead of in
// every commit workgroup.
constexpr int kAppendPlanTables = 1024;
inline bool append_planned(long long B, long long Hkv) { return B * Hkv > kAppendPlanTables; }

struct AllocArgs {
    int p_max;
    long long num_pages;
    int32_t* page_table;
    int32_t* pages;
    int32_t* ring;
    int64_t* ring_ptr;
    uint32_t* status;
    int num_tables;
    const int32_t* demand;
    CallFlags* flags;
    int4* tstate;  // {pages_hi_old, pages_lo_old, ring_off, demand_hi}
};

struct CompactArgs {
    int p_max;
    int T[2];
    long long num_pages;
    int32_t* page_table;
    int32_t* pages;
    int32_t* len;
    int32_t* ring;
    int64_t* ring_ptr;
    int num_tables;
    const uint8_t* release;
    CallFlags* flags;
    int32_t* count;    // [num_tables] released live slots of each table
    int32_t* offset;   // [groups] released slots of each group of group_tables tables
    int group_tables;  // tables per compact_count workgroup
};

// per-table decision of one generation step
enum GenAction : int32_t {
    kGenNone = 0,
    kGenHighVictimToLow = 1,  // candidate stays high; the high victim moves to the low section
    kGenHighVictimOut = 2,    // candidate stays high; the high victim is removed
    kGenCandToLow = 3,        // the candidate moves to the low section
    kGenCandOut = 4           // the candidate is removed
};

struct GenArgs : LayoutArgs {
    uint8_t* pool;
    long long num_pages;
    int32_t* page_table;
    int32_t* pages;
    int32_t* len;
    const int32_t* seq_len;
    int32_t* ring;
    int64_t* ring_ptr;
    uint32_t* status;
    int Hkv, num_tables;
    float alpha_h, alpha_l;
    int window;
    CallFlags* flags;  // ring head/tail before the call; `ok` of the separate plan kernel
    int4* act;         // [num_tables] {action, high index leaving, low index written, 0}
    int4* ids;         // [num_tables] page IDs {leaving token, last high token, low target or -1, 0}
    int32_t* demand;   // [num_tables] bit 0: takes a low page; bit 1: would exceed p_max
    int32_t* offset;   // [num_tables] ring offset of the table's page (separate plan kernel)
};

struct AttnArgs {
    int p_max;
    long long page_bytes;
    long long num_pages;
    int off_kcode[2], off_kmeta[2], off_vcode[2], off_vmeta[2];
    const uint8_t* pool;
    const int32_t* page_table;
    const int32_t* len;
    int B, Hkv, Hq;
    const uint16_t* q;
    float scale_log2;    // sm_scale * log2(e)
    float* out;
    float* lse;
    int splits;          // 0: balanced shares; S >= 1: min(S, pages) ranges per table
    unsigned long long* arrive;  // [T] arrival words of split tables (call tag, count)
    float* part;         // partial states {max, sum, acc[kD]} per head
    int layout;          // index into kLayoutFmts
};

// most shares of the balanced attention mode (sizes its workspace)
constexpr int kAttnMaxWorkers = 2048;

hipError_t launch_append(const AppendArgs& a, int grid_quant, hipStream_t st);
hipError_t launch_alloc(const AllocArgs& a, hipStream_t st);
hipError_t launch_compact(const CompactArgs& a, hipStream_t st);
hipError_t launch_generation(const GenArgs& g, hipStream_t st);
hipError_t launch_attention(AttnArgs a, hipStream_t st);

// Significance update of one decode step: every kept token's score in its page
// becomes the running mean of the softmax probabilities it has received (max
// over the KV head's query heads), from the logits of q and the lse that the
// attention call with the same q wrote.
struct SigArgs {
    int p_max;
    long long num_pages;
    int off_score[2], off_pos[2];
    uint8_t* pool;
    const int32_t* page_table;
    const int32_t* len;
    const int32_t* seq_len;
    int B, Hkv, Hq;
    const uint16_t* q;
    float scale_log2;
    const float* lse;   // [B][Hq] natural log, from the attention call
    int layout;         // index into kLayoutFmts
};
hipError_t launch_significance(const SigArgs& a, hipStream_t st);
// The mode an attention call with `splits` runs in on the current device:
// S >= 1 page ranges per table (S = 1: no split) or -1 (balanced shares);
// *workers = the balanced mode's share count.
hipError_t attention_mode(int gq, int li, long long T, int splits, int* mode, int* workers);

// Prompt-phase significance: rows of q [total_new][Hq][kD] and k
// [total_new][Hkv][kD] concatenated per sequence; score [total_new][Hkv].
struct PromptArgs {
    int B, Hq, Hkv, max_new;
    long long total_new;
    const int32_t* new_len;
    const uint16_t* q;
    const uint16_t* k;
    const float* lse;    // [total_new][Hq] natural log from the caller, or null: the row pass computes it
    float scale_log2;    // sm_scale * log2(e)
    float* score;
    long long* off;      // [B] first row of each sequence (workspace)
    int32_t* nlen;       // [B] rows of each sequence, clamped to max_new and total_new (workspace)
    float* lse2;         // [total_new][Hq] row log2-sum-exp (workspace)
};
hipError_t launch_prompt_significance(const PromptArgs& a, int g, hipStream_t st);

// Fixed device scratch of diffkv_decode_attention_noalloc, one per device.
constexpr long long kNoAllocScratchBytes = 8ll << 20;
hipError_t noalloc_scratch(void** ptr);

}  // namespace dkv
