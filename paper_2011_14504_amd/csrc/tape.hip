// tape.hip -- native replay of a recorded sequence of entry-point calls.
//
// A training step issues a fixed sequence of library calls on a few streams,
// ordered by events, with the same buffers every step.  Recorded once, that
// sequence is replayed here from native code: each call goes through a
// trampoline generated from the entry point's own declaration (every argument
// is carried as a 64-bit word and converted back to the declared parameter
// type), events are tape-owned, and host structures and arrays the calls
// read through pointers are copied into the tape.  Arguments that carry the
// step counter (the stochastic-rounding counter of Eq. 5-6) are rebased on
// every run.
#include <cstring>
#include <new>
#include <string>
#include <type_traits>
#include <utility>
#include <vector>

#include "iseg_common.h"

namespace {

template <typename T>
T from_word(uint64_t w)
{
    if constexpr (std::is_pointer_v<T>) return reinterpret_cast<T>(static_cast<uintptr_t>(w));
    else return static_cast<T>(w);
}

using Tramp = int (*)(void* fn, const uint64_t* w);

template <typename... A, size_t... I>
int call_words(int (*f)(A...), const uint64_t* w, std::index_sequence<I...>)
{
    return f(from_word<A>(w[I])...);
}

template <typename... A>
int tramp(void* f, const uint64_t* w)
{
    return call_words(reinterpret_cast<int (*)(A...)>(f), w, std::index_sequence_for<A...>{});
}

template <typename... A>
constexpr Tramp tramp_of(int (*)(A...)) { return &tramp<A...>; }

template <typename... A>
constexpr int nargs_of(int (*)(A...)) { return (int)sizeof...(A); }

struct Entry {
    const char* name;
    void* fn;
    Tramp call;
    int nargs;
};

#define ISEG_TAPE_ENTRY(f) {#f, (void*)&f, tramp_of(&f), nargs_of(&f)},
const Entry kEntries[] = {
    ISEG_TAPE_ENTRY(iseg_quantize)
    ISEG_TAPE_ENTRY(iseg_requant)
    ISEG_TAPE_ENTRY(iseg_conv_fwd)
    ISEG_TAPE_ENTRY(iseg_conv_bwd_data)
    ISEG_TAPE_ENTRY(iseg_conv_bwd_data_t)
    ISEG_TAPE_ENTRY(iseg_weight_transpose_multi)
    ISEG_TAPE_ENTRY(iseg_conv_bwd_weight)
    ISEG_TAPE_ENTRY(iseg_bn_fwd)
    ISEG_TAPE_ENTRY(iseg_bn_fwd_noalloc)
    ISEG_TAPE_ENTRY(iseg_bn_bwd)
    ISEG_TAPE_ENTRY(iseg_bn_infer)
    ISEG_TAPE_ENTRY(iseg_conv_bn_infer)
    ISEG_TAPE_ENTRY(iseg_bn_fwd_i32)
    ISEG_TAPE_ENTRY(iseg_bn_bwd_i32)
    ISEG_TAPE_ENTRY(iseg_weight_update)
    ISEG_TAPE_ENTRY(iseg_bn_param_update)
    ISEG_TAPE_ENTRY(iseg_update_multi)
    ISEG_TAPE_ENTRY(iseg_weight_quant)
    ISEG_TAPE_ENTRY(iseg_maxpool_fwd)
    ISEG_TAPE_ENTRY(iseg_maxpool_bwd)
    ISEG_TAPE_ENTRY(iseg_sum_requant)
    ISEG_TAPE_ENTRY(iseg_relu_mask_bwd)
    ISEG_TAPE_ENTRY(iseg_sum_requant_relu_mask)
    ISEG_TAPE_ENTRY(iseg_concat_requant)
    ISEG_TAPE_ENTRY(iseg_concat_split)
    ISEG_TAPE_ENTRY(iseg_spatial_sum)
    ISEG_TAPE_ENTRY(iseg_softmax_ce)
    ISEG_TAPE_ENTRY(iseg_mse_onehot)
    ISEG_TAPE_ENTRY(iseg_profile_arm)
    ISEG_TAPE_ENTRY(iseg_status_clear)
    ISEG_TAPE_ENTRY(iseg_check_codes)
};
#undef ISEG_TAPE_ENTRY
constexpr int kNumEntries = (int)(sizeof(kEntries) / sizeof(kEntries[0]));
constexpr int kMaxWords = 32;

enum OpKind { OP_CALL = 0, OP_RECORD = 1, OP_WAIT = 2, OP_ARM = 3 };

struct Op {
    int kind = OP_CALL;
    int entry = -1;                  // OP_CALL / OP_ARM: index into kEntries
    int event = -1;                  // OP_RECORD / OP_WAIT: tape event slot
    int arm = -1;                    // OP_ARM: index among the tape's armed calls
    hipStream_t stream = nullptr;    // OP_RECORD / OP_WAIT
    int step_word = -1;              // word that carries the step counter, or -1
    int64_t step_base = 0;           // that word = step_base + the run's step
    std::vector<uint64_t> words;
    std::vector<uint64_t> blob;      // host data the call reads through pointers (8-byte units)
};

struct Tape {
    std::vector<Op> ops;
    std::vector<hipEvent_t> events;
    int n_arm = 0;
    std::vector<hipEvent_t> arm_events;   // [runs][n_arm][2], empty: the recorded events
    int arm_runs = 0, arm_run = 0;
};

}  // namespace

extern "C" void* iseg_tape_create(void) { return new (std::nothrow) Tape(); }

extern "C" void iseg_tape_destroy(void* t)
{
    Tape* tape = (Tape*)t;
    if (!tape) return;
    for (hipEvent_t e : tape->events) (void)hipEventDestroy(e);
    delete tape;
}

extern "C" int iseg_tape_entry(const char* name)
{
    if (!name) return -1;
    for (int i = 0; i < kNumEntries; i++)
        if (std::strcmp(kEntries[i].name, name) == 0) return i;
    return -1;
}

extern "C" int iseg_tape_entry_nargs(int entry)
{
    return entry >= 0 && entry < kNumEntries ? kEntries[entry].nargs : -1;
}

extern "C" int iseg_tape_add_call(void* t, int entry, const uint64_t* words, int n_words, const void* blob,
                                  size_t blob_bytes, const int32_t* blob_words, int n_blob_words,
                                  int32_t step_word, int64_t step_base)
{
    Tape* tape = (Tape*)t;
    if (!tape || entry < 0 || entry >= kNumEntries || n_words != kEntries[entry].nargs || n_words > kMaxWords ||
        (n_words && !words) || (blob_bytes && !blob) || (n_blob_words && !blob_words) || blob_bytes % 8 ||
        step_word < -1 || step_word >= n_words)
        return ISEG_ERR_ARG;
    Op op;
    op.entry = entry;
    op.words.assign(words, words + n_words);
    op.blob.resize(blob_bytes / 8);
    if (blob_bytes) std::memcpy(op.blob.data(), blob, blob_bytes);
    // blob words hold byte offsets into the blob: make them addresses of the
    // tape's copy (its storage never moves again)
    for (int i = 0; i < n_blob_words; i++) {
        const int k = blob_words[i];
        if (k < 0 || k >= n_words || op.words[k] >= blob_bytes) return ISEG_ERR_ARG;
        op.words[k] = (uint64_t)(uintptr_t)((const char*)op.blob.data() + op.words[k]);
    }
    op.step_word = step_word;
    op.step_base = step_base;
    if (std::strcmp(kEntries[entry].name, "iseg_profile_arm") == 0) {
        op.kind = OP_ARM;
        op.arm = tape->n_arm++;
    }
    tape->ops.push_back(std::move(op));
    return ISEG_OK;
}

static int tape_event(Tape* tape, int slot)
{
    if (slot < 0 || slot > (1 << 20)) return ISEG_ERR_ARG;
    while ((int)tape->events.size() <= slot) {
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return ISEG_ERR_DEVICE;
        tape->events.push_back(e);
    }
    return ISEG_OK;
}

extern "C" int iseg_tape_add_record(void* t, int32_t slot, hipStream_t stream)
{
    Tape* tape = (Tape*)t;
    if (!tape) return ISEG_ERR_ARG;
    int rc = tape_event(tape, slot);
    if (rc) return rc;
    Op op;
    op.kind = OP_RECORD;
    op.event = slot;
    op.stream = stream;
    tape->ops.push_back(std::move(op));
    return ISEG_OK;
}

extern "C" int iseg_tape_add_wait(void* t, hipStream_t stream, int32_t slot)
{
    Tape* tape = (Tape*)t;
    if (!tape) return ISEG_ERR_ARG;
    int rc = tape_event(tape, slot);
    if (rc) return rc;
    Op op;
    op.kind = OP_WAIT;
    op.event = slot;
    op.stream = stream;
    tape->ops.push_back(std::move(op));
    return ISEG_OK;
}

extern "C" int iseg_tape_arm_count(const void* t) { return t ? ((const Tape*)t)->n_arm : -1; }

extern "C" int iseg_tape_set_arm_events(void* t, const hipEvent_t* events, int32_t runs)
{
    Tape* tape = (Tape*)t;
    if (!tape || runs < 0 || (runs && !events)) return ISEG_ERR_ARG;
    tape->arm_events.assign(events, events + (size_t)runs * tape->n_arm * 2);
    tape->arm_runs = runs;
    tape->arm_run = 0;
    return ISEG_OK;
}

extern "C" int iseg_tape_run(void* t, uint32_t step, int64_t* failed_op)
{
    Tape* tape = (Tape*)t;
    if (failed_op) *failed_op = -1;
    if (!tape) return ISEG_ERR_ARG;
    const bool arm_sub = tape->arm_runs > 0 && tape->arm_run < tape->arm_runs;
    uint64_t w[kMaxWords];
    for (size_t i = 0; i < tape->ops.size(); i++) {
        const Op& op = tape->ops[i];
        int rc = ISEG_OK;
        if (op.kind == OP_RECORD) {
            rc = hipEventRecord(tape->events[op.event], op.stream) == hipSuccess ? ISEG_OK : ISEG_ERR_DEVICE;
        } else if (op.kind == OP_WAIT) {
            rc = hipStreamWaitEvent(op.stream, tape->events[op.event], 0) == hipSuccess ? ISEG_OK : ISEG_ERR_DEVICE;
        } else {
            if (op.kind == OP_ARM && !arm_sub) continue;     // armed slots fire only with caller events
            const size_t n = op.words.size();
            std::memcpy(w, op.words.data(), n * sizeof(uint64_t));
            if (op.step_word >= 0) w[op.step_word] = (uint64_t)(op.step_base + (int64_t)step);
            if (op.kind == OP_ARM) {
                const size_t k = ((size_t)tape->arm_run * tape->n_arm + op.arm) * 2;
                w[1] = (uint64_t)(uintptr_t)tape->arm_events[k];
                w[2] = (uint64_t)(uintptr_t)tape->arm_events[k + 1];
            }
            rc = kEntries[op.entry].call(kEntries[op.entry].fn, w);
        }
        if (rc != ISEG_OK) {
            if (failed_op) *failed_op = (int64_t)i;
            return rc;
        }
    }
    if (arm_sub) tape->arm_run++;
    return ISEG_OK;
}

extern "C" int64_t iseg_tape_size(const void* t) { return t ? (int64_t)((const Tape*)t)->ops.size() : -1; }
