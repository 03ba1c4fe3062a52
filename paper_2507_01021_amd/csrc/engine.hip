// Engine: device weights, caches and workspaces of one context, and the
// encode pass / decode step that drive the kernels on the context's stream.
//
// Encode pass (Listing 1: features per segment, pad to 30 s, stack, encode):
//   audio -> reflect-padded window -> DFT power (fp32 matrix cores, window
//   folded into the basis) -> mel projection + log10 (fp32 matrix cores) ->
//   per-segment max and normalisation -> conv stem (two implicit-im2col
//   GEMMs over overlapping rows) -> encoder layers (LN, QK and V
//   projections, attention, output projection + residual, LN, fc1 + GELU,
//   fc2 + residual) -> final LN -> cross-attention keys and values of every
//   decoder layer written straight into the slots' caches -> prompts seated
//   (and, with prefill, prompt positions 0..n_prompt-2 run through the
//   decoder layers).
// Decode step (greedy generate, one token per active slot):
//   embedding -> per layer: LN, fused QKV projection appending this position
//   to the self-attention cache, self-attention over the slot's positions,
//   output projection + residual, LN, cross query, cross-attention over the
//   1500 cached encoder positions, output projection +
//   residual, LN, fc1 + GELU, fc2 + residual -> final LN -> logits against
//   the token embedding -> argmax, next input, position advance.
//   In bf16 the projection weights and the activations they multiply are
//   fragment-major (frag_off). With 32 or more slots in bf16 the rows are
//   split in two halves (the first a whole number of 16-row tiles) that run
//   the complete step on two streams, each as its own captured graph (the
//   halves touch disjoint slots), so the two chains of small latency-bound
//   kernels overlap. While the slot list stays the same the chains are not
//   joined between steps (one may run a step ahead of the other); any other
//   call joins them first. Steps with decode-kernel timing on run unsplit, so
//   each timed launch has the device to itself.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <map>
#include <mutex>
#include <type_traits>
#include <string>
#include <vector>

#include "engine.h"
#include "kernels.h"

namespace wmi {

// ------------------------------------------------------------------ blob

struct TensorSpec {
    std::string name;
    std::vector<long long> shape;
    long long numel() const {
        long long n = 1;
        for (auto s : shape) n *= s;
        return n;
    }
};

static void add_attn(std::vector<TensorSpec>& v, const std::string& p, long long d) {
    v.push_back({p + ".q.w", {d, d}});
    v.push_back({p + ".q.b", {d}});
    v.push_back({p + ".k.w", {d, d}});
    v.push_back({p + ".v.w", {d, d}});
    v.push_back({p + ".v.b", {d}});
    v.push_back({p + ".o.w", {d, d}});
    v.push_back({p + ".o.b", {d}});
}
static void add_ln(std::vector<TensorSpec>& v, const std::string& p, long long d) {
    v.push_back({p + ".g", {d}});
    v.push_back({p + ".b", {d}});
}
static void add_mlp(std::vector<TensorSpec>& v, const std::string& p, long long d) {
    v.push_back({p + ".fc1.w", {4 * d, d}});
    v.push_back({p + ".fc1.b", {4 * d}});
    v.push_back({p + ".fc2.w", {d, 4 * d}});
    v.push_back({p + ".fc2.b", {d}});
}

static std::vector<TensorSpec> canonical_specs(const whisper_params& p) {
    const long long d = p.n_audio_state;
    std::vector<TensorSpec> v;
    v.push_back({"enc.conv1.w", {d, p.n_mels, 3}});
    v.push_back({"enc.conv1.b", {d}});
    v.push_back({"enc.conv2.w", {d, d, 3}});
    v.push_back({"enc.conv2.b", {d}});
    for (int i = 0; i < p.n_audio_layer; ++i) {
        const std::string q = "enc." + std::to_string(i);
        add_ln(v, q + ".attn_ln", d);
        add_attn(v, q + ".attn", d);
        add_ln(v, q + ".mlp_ln", d);
        add_mlp(v, q + ".mlp", d);
    }
    add_ln(v, "enc.ln_post", d);
    if (p.n_text_layer == 0) {  // encoder-only CTC model: the head instead of a decoder
        v.push_back({"ctc.w", {p.n_vocab, d}});
        v.push_back({"ctc.b", {p.n_vocab}});
        return v;
    }
    v.push_back({"dec.tok_emb", {p.n_vocab, d}});
    v.push_back({"dec.pos_emb", {p.n_text_ctx, d}});
    for (int i = 0; i < p.n_text_layer; ++i) {
        const std::string q = "dec." + std::to_string(i);
        add_ln(v, q + ".attn_ln", d);
        add_attn(v, q + ".attn", d);
        add_ln(v, q + ".cross_ln", d);
        add_attn(v, q + ".cross", d);
        add_ln(v, q + ".mlp_ln", d);
        add_mlp(v, q + ".mlp", d);
    }
    add_ln(v, "dec.ln", d);
    return v;
}

static size_t blob_size(const whisper_params& p, std::map<std::string, std::pair<size_t, long long>>* offs) {
    const size_t esz = p.dtype == WHISPER_DTYPE_F32 ? 4 : 2;
    size_t off = 256;
    for (auto& t : canonical_specs(p)) {
        if (offs) (*offs)[t.name] = {off, t.numel()};
        off += (size_t)t.numel() * esz;
        off = (off + 255) / 256 * 256;
    }
    return off;
}

int parse_blob_header(const void* blob, size_t bytes, whisper_params* out, const char** why) {
    if (!blob || bytes < 256) { *why = "blob shorter than its 256-byte header"; return WHISPER_E_FORMAT; }
    const char* b = static_cast<const char*>(blob);
    if (memcmp(b, "WHSPMI01", 8) != 0) { *why = "bad blob magic"; return WHISPER_E_FORMAT; }
    int32_t h[14];
    memcpy(h, b + 8, sizeof(h));
    if (h[0] != 1) { *why = "unsupported blob version"; return WHISPER_E_FORMAT; }
    whisper_params p;
    memset(&p, 0, sizeof(p));
    p.dtype = h[1];
    p.n_mels = h[2]; p.n_audio_ctx = h[3]; p.n_audio_state = h[4]; p.n_audio_head = h[5];
    p.n_audio_layer = h[6]; p.n_vocab = h[7]; p.n_text_ctx = h[8]; p.n_text_state = h[9];
    p.n_text_head = h[10]; p.n_text_layer = h[11];
    p.max_slots = 32;
    *out = p;
    return WHISPER_OK;
}

// ------------------------------------------------------------------ tables (host, double)

constexpr double kPi = 3.14159265358979323846;

// k-major [400][DFT_ROWS]: column 2k, 2k+1 = w cos, w sin of bin k at sample n
// (periodic Hann w), columns 402 .. DFT_ROWS-1 zero
static std::vector<float> dft_basis() {
    std::vector<float> b(400 * DFT_ROWS, 0.f);
    for (int k = 0; k <= 200; ++k)
        for (int n = 0; n < 400; ++n) {
            const double w = 0.5 - 0.5 * cos(2.0 * kPi * n / 400.0);
            const double ang = 2.0 * kPi * (double)((k * n) % 400) / 400.0;
            b[n * DFT_ROWS + 2 * k] = (float)(w * cos(ang));
            b[n * DFT_ROWS + 2 * k + 1] = (float)(w * sin(ang));
        }
    return b;
}

static double slaney_mel(double f) {
    return f < 1000.0 ? 3.0 * f / 200.0 : 15.0 + log(f / 1000.0) / (log(6.4) / 27.0);
}
static double slaney_hz(double m) {
    return m < 15.0 ? 200.0 * m / 3.0 : 1000.0 * exp((m - 15.0) * (log(6.4) / 27.0));
}

static std::vector<float> mel_bank(int nm) {  // [nm][201]
    std::vector<double> edges(nm + 2);
    const double top = slaney_mel(8000.0);
    for (int i = 0; i < nm + 2; ++i) edges[i] = slaney_hz(top * i / (nm + 1));
    std::vector<float> fb((size_t)nm * 201);
    for (int i = 0; i < nm; ++i)
        for (int k = 0; k < 201; ++k) {
            const double f = 40.0 * k;
            const double up = (f - edges[i]) / (edges[i + 1] - edges[i]);
            const double down = (edges[i + 2] - f) / (edges[i + 2] - edges[i + 1]);
            const double tri = std::max(0.0, std::min(up, down));
            fb[(size_t)i * 201 + k] = (float)(tri * 2.0 / (edges[i + 2] - edges[i]));
        }
    return fb;
}

static std::vector<float> sinusoids(int T, int d) {  // [T][d]
    std::vector<float> pe((size_t)T * d);
    const int half = d / 2;
    const double inc = log(10000.0) / (half - 1);
    for (int t = 0; t < T; ++t)
        for (int j = 0; j < half; ++j) {
            const double a = t * exp(-inc * j);
            pe[(size_t)t * d + j] = (float)sin(a);
            pe[(size_t)t * d + half + j] = (float)cos(a);
        }
    return pe;
}

// ------------------------------------------------------------------ scratch of the allocation-free step
//
// whisper_batch_decode_step_noalloc keeps its per-step temporaries (slot
// list, row lengths, activations, split-K partial sums, greedy-choice keys,
// tokens, and the fp32 model's logits) in this array instead of the
// context's workspaces. Each GPU holds its own copy until the process ends.
// In host code `scratch` only names the symbol: its device address on a
// device comes from hipGetSymbolAddress with that device current, taken once
// per device when an engine is created there and kept in g_scratch_dev.
static __device__ __align__(256) unsigned char scratch[WHISPER_NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
constexpr int MAX_DEVICES = 64;
void* g_scratch_dev[MAX_DEVICES] = {};
}  // namespace

// Device address of `scratch` on device dev (the current device).
static void* scratch_address(int dev) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (dev < 0 || dev >= MAX_DEVICES) throw ArgError(WHISPER_E_INVAL, "device index above 63");
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        WMI_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        g_scratch_dev[dev] = p;
    }
    return g_scratch_dev[dev];
}

// A slot list passed by value, so that staging it needs no copy from host memory.
struct RowList {
    int n;
    int slot[WHISPER_NOALLOC_MAX_ROWS];
};
__global__ void put_list_kernel(RowList l, int* __restrict__ dst) {
    if ((int)threadIdx.x < l.n) dst[threadIdx.x] = l.slot[threadIdx.x];
}

// ------------------------------------------------------------------ engine

template <class T> struct HostElem;
template <> struct HostElem<float> { static float to_f(const void* p, long long i) { return static_cast<const float*>(p)[i]; } };
template <> struct HostElem<bf16> {
    static float to_f(const void* p, long long i) { bf16 v; v.x = static_cast<const uint16_t*>(p)[i]; return bf2f(v); }
};

template <class T>
struct EncLayerW {
    float *ln1g, *ln1b, *bq, *bv, *bo, *ln2g, *ln2b, *b1, *b2;
    T *Wqk, *Wv, *Wo, *W1, *W2;
};
template <class T>
struct DecLayerW {
    float *ln1g, *ln1b, *bq, *bv, *bo, *ln2g, *ln2b, *cbq, *cbo, *ln3g, *ln3b, *b1, *b2;
    T *Wqkv, *Wo, *Wcq, *Wco, *W1, *W2;
};


template <class T>
class EngineT final : public Engine {
   public:
    EngineT(const whisper_params& p, const void* blob, size_t bytes, int device)
        : P_(p), dev_(device) {
        d_ = p.n_audio_state; H_ = p.n_audio_head; Le_ = p.n_audio_layer; Ld_ = p.n_text_layer;
        V_ = p.n_vocab; nm_ = p.n_mels; S_ = p.max_slots;
        EB_ = p.max_encode_batch;
        ctc_ = Ld_ == 0;
        prefill_ = !ctc_ && p.prefill != 0;
        WMI_HIP(hipSetDevice(dev_));
        WMI_HIP(hipStreamCreateWithFlags(&own_stream_, hipStreamNonBlocking));
        for (int c = 1; c < MAXC; ++c) {
            WMI_HIP(hipStreamCreateWithFlags(&cst_[c], hipStreamNonBlocking));
            WMI_HIP(hipEventCreateWithFlags(&join_ev_[c], hipEventDisableTiming));
        }
        WMI_HIP(hipEventCreateWithFlags(&fork_ev_, hipEventDisableTiming));
        for (int k = 0; k < ENC_PARTS_MAX - 1; ++k) {
            WMI_HIP(hipStreamCreateWithFlags(&es_[k], hipStreamNonBlocking));
            WMI_HIP(hipEventCreateWithFlags(&enc_join_[k], hipEventDisableTiming));
        }
        WMI_HIP(hipEventCreateWithFlags(&enc_fork_, hipEventDisableTiming));
        st_ = own_stream_;
        if (const char* g = getenv("WHISPER_STEP_GRAPHS")) graphs_ = g[0] != '0';
        if (const char* g = getenv("WHISPER_STEP_SPLIT")) split_ = g[0] != '0';
        if (const char* g = getenv("WHISPER_STEP_CHAINS")) chains_ = std::max(1, std::min(MAXC, atoi(g)));
        if (const char* g = getenv("WHISPER_FUSED_LN")) fused_ln_ = g[0] != '0';
        if (const char* g = getenv("WHISPER_FREE_CHAINS")) free_run_ = g[0] != '0';
        if (const char* g = getenv("WHISPER_FC2_SPLIT")) fc2_split_ = atoi(g);
        if (const char* g = getenv("WHISPER_ENC_SPLIT")) enc_parts_ = std::max(1, std::min(ENC_PARTS_MAX, atoi(g)));
        load_weights(blob, bytes);
        alloc_state();
        scratch_ = static_cast<unsigned char*>(scratch_address(dev_));
        WMI_HIP(hipDeviceSynchronize());
    }

    ~EngineT() override {
        (void)hipSetDevice(dev_);
        if (st_) (void)hipStreamSynchronize(st_);
        for (auto q : es_)
            if (q) (void)hipStreamSynchronize(q);
        if (ctc_st_) (void)hipStreamSynchronize(ctc_st_);
        for (auto& pr : prof_)
            for (auto& e : pr.used) { (void)hipEventDestroy(e.first); (void)hipEventDestroy(e.second); }
        for (auto e : event_pool_) (void)hipEventDestroy(e);
        for (auto e : marks_) (void)hipEventDestroy(e);
        if (mark_start_) (void)hipEventDestroy(mark_start_);
        for (int c = 1; c < MAXC; ++c)
            if (cst_[c]) (void)hipStreamSynchronize(cst_[c]);
        for (auto* m : {&step_graphs_, &stamped_graphs_})
            for (auto& g : *m)
                for (auto ge : g.second)
                    if (ge) (void)hipGraphExecDestroy(ge);
        for (auto& s : stage_) {
            if (s.ev) (void)hipEventDestroy(s.ev);
            if (s.host) (void)hipHostFree(s.host);
        }
        if (tokpin_) (void)hipHostFree(tokpin_);
        for (int b = 0; b < 2; ++b) {
            if (stop_pin_[b]) (void)hipHostFree(stop_pin_[b]);
            if (stop_ev_[b]) (void)hipEventDestroy(stop_ev_[b]);
        }
        for (void* q : allocs_) (void)hipFree(q);
        if (fork_ev_) (void)hipEventDestroy(fork_ev_);
        for (int c = 1; c < MAXC; ++c) {
            if (join_ev_[c]) (void)hipEventDestroy(join_ev_[c]);
            if (cst_[c]) (void)hipStreamDestroy(cst_[c]);
        }
        for (int q = 0; q < 2; ++q) {
            if (ctc_head_[q]) (void)hipEventDestroy(ctc_head_[q]);
            if (ctc_done_[q]) (void)hipEventDestroy(ctc_done_[q]);
        }
        if (ctc_st_) (void)hipStreamDestroy(ctc_st_);
        if (enc_fork_) (void)hipEventDestroy(enc_fork_);
        for (int k = 0; k < ENC_PARTS_MAX - 1; ++k) {
            if (enc_join_[k]) (void)hipEventDestroy(enc_join_[k]);
            if (es_[k]) (void)hipStreamDestroy(es_[k]);
        }
        if (own_stream_) (void)hipStreamDestroy(own_stream_);
    }

    void set_stream(void* s) override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        st_ = s ? static_cast<hipStream_t>(s) : own_stream_;
    }

    void sync() override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        if (ctc_st_) WMI_HIP(hipStreamSynchronize(ctc_st_));
    }

    // -------------------------------------------------------------- encode
    void encode(const SegmentDesc* segs, int n, const int* slots, bool sync_) override {
        join_chains();
        WMI_HIP(hipSetDevice(dev_));
        for (int s0 = 0; s0 < n; s0 += EB_) encode_pass(segs + s0, std::min(EB_, n - s0), slots + s0);
        WMI_HIP(hipGetLastError());
        if (sync_) WMI_HIP(hipStreamSynchronize(st_));
    }

    // Steps of an unchanged slot list may leave the chains running apart
    // (each on its own stream, ahead or behind the others); everything else
    // first joins them into the context's stream.
    void join_chains() {
        if (!chains_apart_) return;
        for (int c = 1; c < apart_nc_; ++c) {
            WMI_HIP(hipEventRecord(join_ev_[c], cst_[c]));
            WMI_HIP(hipStreamWaitEvent(st_, join_ev_[c], 0));
        }
        chains_apart_ = false;
    }

    // -------------------------------------------------------------- decode step
    void decode_step(const int* slots, int n, const int* forced, int* out_tok, float* out_logits,
                     bool sync_) override {
        WMI_HIP(hipSetDevice(dev_));
        const bool same_list = n == (int)list_host_.size() && std::equal(slots, slots + n, list_host_.begin());
        // timing of a decode kernel (or of the whole step) brackets each launch
        // with events: such steps run as plain launches, unsplit; encoder
        // timings leave the steps as they are
        const bool timed = prof_[WHISPER_K_CROSS_ATTN].on || prof_[WHISPER_K_SELF_ATTN].on || prof_[WHISPER_K_DEC_STEP].on;
        // cross-attention spans stamped inside the plain steps' graphs: graphs and
        // chains as usual, but the chains are joined and read after every step
        const bool stamping = prof_[WHISPER_K_CROSS_ATTN_STEP].on;
        const bool plain = graphs_ && !forced && !out_tok && !out_logits && !timed && !sync_ && !stamping;
        if (free_run_ && plain && same_list && chains_apart_) {
            // the chains keep running on their own streams: no fork, no join
            auto it = step_graphs_.find(n);
            if (it != step_graphs_.end()) {
                for (int c = 0; c < apart_nc_; ++c) WMI_HIP(hipGraphLaunch(it->second[c], c == 0 ? st_ : cst_[c]));
                WMI_HIP(hipGetLastError());
                return;
            }
        }
        join_chains();
        if (!same_list) {
            list_host_.assign(slots, slots + n);
            upload(0, list_, slots, n * sizeof(int));
        }
        if (forced) upload(1, forced_, forced, n * sizeof(int));
        // Plain steps (no teacher forcing, no per-step outputs, no kernel
        // timing) replay captured graphs of the whole step; a graph only
        // depends on the row count because the slot list lives in device memory.
        int r0[MAXC + 1];
        const int nc = timed ? (r0[0] = 0, r0[1] = n, 1) : chain_rows(n, r0);
        auto stream = [&](int c) { return c == 0 ? st_ : cst_[c]; };
        prof_begin(WHISPER_K_DEC_STEP, st_);
        if (nc > 1) {  // fork: every chain waits for everything enqueued so far
            WMI_HIP(hipEventRecord(fork_ev_, st_));
            for (int c = 1; c < nc; ++c) WMI_HIP(hipStreamWaitEvent(cst_[c], fork_ev_, 0));
        }
        stamp_on_ = stamping;
        if (graphs_ && !forced && !out_tok && !out_logits && !timed) {
            auto& graphs = stamping ? stamped_graphs_ : step_graphs_;
            auto it = graphs.find(n);
            if (it == graphs.end()) {
                std::array<hipGraphExec_t, MAXC> ge{};
                for (int c = 0; c < nc; ++c)
                    ge[c] = capture(stream(c), [&] { launch_rows(r0[c], r0[c + 1] - r0[c], false, false, stream(c), c); });
                it = graphs.emplace(n, ge).first;
            }
            for (int c = 0; c < nc; ++c) WMI_HIP(hipGraphLaunch(it->second[c], stream(c)));
        } else {
            for (int c = 0; c < nc; ++c)
                launch_rows(r0[c], r0[c + 1] - r0[c], forced != nullptr, out_logits != nullptr, stream(c), c);
        }
        stamp_on_ = false;
        if (free_run_ && plain && nc > 1) {  // stay apart until something needs the results
            chains_apart_ = true;
            apart_nc_ = nc;
        } else {
            for (int c = 1; c < nc; ++c) {  // join
                WMI_HIP(hipEventRecord(join_ev_[c], cst_[c]));
                WMI_HIP(hipStreamWaitEvent(st_, join_ev_[c], 0));
            }
        }
        prof_end(WHISPER_K_DEC_STEP, st_);
        WMI_HIP(hipGetLastError());
        if (stamping) read_stamps(nc);
        if (out_tok) WMI_HIP(hipMemcpyAsync(out_tok, outtok_, n * sizeof(int), hipMemcpyDeviceToHost, st_));
        if (out_logits)
            WMI_HIP(hipMemcpyAsync(out_logits, logits_, (size_t)n * V_ * sizeof(float), hipMemcpyDeviceToHost, st_));
        if (sync_ || out_tok || out_logits || forced) {
            WMI_HIP(hipStreamSynchronize(st_));
            check_decode_error();
        }
    }

    // Rows of a step of n rows cut into chains (independent launch
    // sequences on their own streams): one chain below 32 rows (or in fp32),
    // else up to chains_ chains of whole 16-row tiles, as even as the tiles
    // allow. r0[c] .. r0[c + 1] - 1 are chain c's rows; returns the count.
    int chain_rows(int n, int* r0) const {
        const int tiles = (n + 15) / 16;
        const int k = (!split_ || !std::is_same<T, bf16>::value || n < 32) ? 1 : std::min(chains_, tiles);
        r0[0] = 0;
        for (int c = 1; c < k; ++c)  // boundary c: the tile nearest c * n / k, one tile per chain at least
            r0[c] = 16 * std::max(r0[c - 1] / 16 + 1, std::min(tiles - (k - c), (2 * c * n + 16 * k) / (32 * k)));
        r0[k] = n;
        return k;
    }

    template <class F>
    hipGraphExec_t capture(hipStream_t s, F&& launches) {
        hipGraph_t g = nullptr;
        hipGraphExec_t ge = nullptr;
        WMI_HIP(hipStreamBeginCapture(s, hipStreamCaptureModeRelaxed));
        launches();
        WMI_HIP(hipStreamEndCapture(s, &g));
        const hipError_t e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
        (void)hipGraphDestroy(g);
        WMI_HIP(e);
        return ge;
    }

    // Device buffers of a set of decoder rows: the slot (and, for prefill
    // rows, the position) of each row, the activations and the split-K
    // partial sums.
    struct RowBufs {
        const int* list;
        const int* rowpos;  // null: each row is at its slot's current position
        float* dx;
        T* dz;
        T* dq;
        T* datt;
        T* dh;
        int* rowlen;
        float* pbuf;
        unsigned long long* stamps = nullptr;  // cross-attention timing slots [layer][2], or null
    };

    // Embedding and every decoder layer for n rows; leaves the final layer
    // norm of each row in b.dz.
    void decoder_layers(const RowBufs& b, int n, hipStream_t s) {
        const int d = d_;
        const int ks1 = split_k(d);
        const int ks4 = fc2_split_ == 8 && (4 * d / 32) % 8 == 0 ? 8 : split_k(4 * d);
        WMI_SWITCH_E(d, hipLaunchKernelGGL((embed_ln_kernel<T, E>), dim3(n), dim3(64), 0, s, tok_emb_, pos_emb_,
                                           b.list, pos_, b.rowpos, seq_, b.dx, b.dz, dec_[0].ln1g, dec_[0].ln1b));
        for (int l = 0; l < Ld_; ++l) {
            const DecLayerW<T>& L = dec_[l];
            const long long sl = (long long)l * S_ * H_ * 64;
            proj(L.Wqkv, 3 * d, b.dz, n, d, 1,
                 EpiDecQKV<T>{L.bq, L.bv, b.dq, kts_ + sl * TS, vs_ + sl * TS, b.list, pos_, b.rowpos, b.rowlen, d,
                              H_},
                 s);
            DecAttnArgs sa{b.dq, kts_ + sl * TS, vs_ + sl * TS, b.datt, b.list, b.rowlen, TS, H_, d};
            prof_begin(WHISPER_K_SELF_ATTN, s);
            if constexpr (std::is_same<T, bf16>::value)
                hipLaunchKernelGGL(self_attn_bf16_kernel, dim3(H_, n), dim3(256), 0, s, sa);
            else
                hipLaunchKernelGGL(self_attn_kernel<T>, dim3(H_, n), dim3(256), 0, s, sa);
            prof_end(WHISPER_K_SELF_ATTN, s);
            self_out_cross_q(L, n, b.datt, b.dq, b.dx, b.dz, b.pbuf, s);
            DecAttnArgs ca{b.dq, ktc_ + sl * TC, vc_ + sl * TC, b.datt, b.list, nullptr, TC, H_, d,
                           b.stamps ? b.stamps + 2 * l : nullptr};
            prof_begin(WHISPER_K_CROSS_ATTN, s);
            hipLaunchKernelGGL(cross_attn_kernel<T>, dim3(H_, n), dim3(64 * CW), 0, s, ca);
            prof_end(WHISPER_K_CROSS_ATTN, s);
            proj_resid(L.Wco, b.datt, n, d, ks1, L.cbo, L.ln3g, L.ln3b, b.pbuf, b.dx, b.dz, s);
            proj(L.W1, 4 * d, b.dz, n, d, 1, EpiGelu<T, true>{L.b1, b.dh, 4 * d}, s);
            const bool last = l + 1 == Ld_;
            proj_resid(L.W2, b.dh, n, 4 * d, ks4, L.b2, last ? lnfg_ : dec_[l + 1].ln1g,
                       last ? lnfb_ : dec_[l + 1].ln1b, b.pbuf, b.dx, b.dz, s);
        }
    }

    // The kernels of one decode step for rows r0 .. r0+n-1 of the slot list,
    // on stream s, with chain c's split-K partial buffer. r0 is a multiple
    // of 16, so the fragment-major activations of these rows start at
    // element r0 * K.
    void launch_rows(int r0, int n, bool forced, bool want_logits, hipStream_t s, int c) {
        const int d = d_;
        unsigned long long* stamps = nullptr;
        if (stamp_on_) {  // this chain's slots: one (start, end) pair per layer, reset first
            stamps = stamps_ + (size_t)c * Ld_ * 2;
            hipLaunchKernelGGL(stamp_reset_kernel, dim3((Ld_ + 63) / 64), dim3(64), 0, s, stamps, Ld_);
        }
        const StepBufs b{RowBufs{list_ + r0, nullptr, dx_ + (size_t)r0 * d, dz_ + (size_t)r0 * d,
                                 dq_ + (size_t)r0 * d, datt_ + (size_t)r0 * d, dh_ + (size_t)r0 * 4 * d,
                                 rowlen_ + r0, gpart_ + (size_t)c * KSMAX * S_ * d, stamps},
                         logits_ + (size_t)r0 * V_, keys_ + (size_t)r0 * nkeys_, outtok_ + r0,
                         forced ? forced_ + r0 : nullptr};
        run_step(b, n, want_logits, s);
    }

    // Buffers of one step's rows: the decoder rows, the logits (fp32 model:
    // always written; bf16: when asked for), greedy-choice keys, tokens out
    // and forced tokens in (or null).
    struct StepBufs {
        RowBufs rows;
        float* logits;
        unsigned long long* keys;
        int* outtok;
        const int* forced;
    };

    // Every kernel of one decode step for n rows, on stream s.
    void run_step(const StepBufs& sb, int n, bool want_logits, hipStream_t s) {
        const int d = d_;
        const RowBufs& b = sb.rows;
        decoder_layers(b, n, s);
        const int* list = b.list;
        float* logits = sb.logits;
        unsigned long long* keys = sb.keys;
        const TokenFilter tf{use_never_ ? never_mask_ : nullptr, use_first_ ? first_mask_ : nullptr, list, pos_, npr_};
        int nk = ARGMAX_CHUNKS;
        if constexpr (std::is_same<T, bf16>::value) {
            // the head kernel keeps one key per row and workgroup; logits only when asked for
            nk = head_argmax(tok_emb_, V_, b.dz, n, d, HeadArgs{want_logits ? logits : nullptr, keys, V_, tf}, s);
        } else {
            proj(tok_emb_, V_, b.dz, n, d, 1, EpiLogits{logits, V_}, s);
            hipLaunchKernelGGL(argmax_keys_kernel, dim3(ARGMAX_CHUNKS, n), dim3(256), 0, s, logits, V_, keys, tf);
        }
        hipLaunchKernelGGL(argmax_step_kernel, dim3(n), dim3(64), 0, s, keys, nk, list, pos_, npr_, seq_, gen_,
                           sb.forced, sb.outtok, eot_, stop_at_, dec_err_);
    }

    // Scratch layout of an allocation-free step of n rows (byte offsets,
    // each region 256-byte aligned); total() is what the array must hold.
    struct NoallocLayout {
        size_t list, rowlen, outtok, dx, dz, dq, datt, dh, part, keys, logits, end;
    };
    NoallocLayout noalloc_layout(int n) const {
        const size_t d = d_, n16 = (size_t)(n + 15) / 16 * 16;
        size_t o = 0;
        auto take = [&](size_t bytes) { const size_t at = o; o += (bytes + 255) / 256 * 256; return at; };
        NoallocLayout L;
        L.list = take(WHISPER_NOALLOC_MAX_ROWS * sizeof(int));
        L.rowlen = take(WHISPER_NOALLOC_MAX_ROWS * sizeof(int));
        L.outtok = take(WHISPER_NOALLOC_MAX_ROWS * sizeof(int));
        L.dx = take((size_t)n * d * sizeof(float));
        L.dz = take(n16 * d * sizeof(T));
        L.dq = take((size_t)n * d * sizeof(T));
        L.datt = take(n16 * d * sizeof(T));
        L.dh = take(n16 * 4 * d * sizeof(T));
        L.part = take((size_t)KSMAX * n * d * sizeof(float));
        L.keys = take((size_t)n * nkeys_ * sizeof(unsigned long long));
        L.logits = std::is_same<T, bf16>::value ? o : take((size_t)n * V_ * sizeof(float));
        L.end = o;
        return L;
    }

    void decode_step_noalloc(const int* slots, int n, int* out_tok_dev) override {
        if (n < 1 || n > WHISPER_NOALLOC_MAX_ROWS)
            throw ArgError(WHISPER_E_CAPACITY, "decode_step_noalloc: n must be in 1.." +
                                                   std::to_string(WHISPER_NOALLOC_MAX_ROWS));
        const NoallocLayout L = noalloc_layout(n);
        if (L.end > (size_t)WHISPER_NOALLOC_SCRATCH_BYTES)
            throw ArgError(WHISPER_E_CAPACITY, "decode_step_noalloc: " + std::to_string(n) + " rows of this model need " +
                                                   std::to_string(L.end) + " bytes of scratch, the array holds " +
                                                   std::to_string((size_t)WHISPER_NOALLOC_SCRATCH_BYTES));
        for (auto& pr : prof_)
            if (pr.on) throw ArgError(WHISPER_E_STATE, "decode_step_noalloc: kernel timing is on");
        WMI_HIP(hipSetDevice(dev_));
        join_chains();
        unsigned char* z = scratch_;  // this device's copy of the array
        RowList rl;
        rl.n = n;
        for (int i = 0; i < n; ++i) rl.slot[i] = slots[i];
        int* list = reinterpret_cast<int*>(z + L.list);
        hipLaunchKernelGGL(put_list_kernel, dim3(1), dim3(WHISPER_NOALLOC_MAX_ROWS), 0, st_, rl, list);
        const StepBufs b{RowBufs{list, nullptr, reinterpret_cast<float*>(z + L.dx), reinterpret_cast<T*>(z + L.dz),
                                 reinterpret_cast<T*>(z + L.dq), reinterpret_cast<T*>(z + L.datt),
                                 reinterpret_cast<T*>(z + L.dh), reinterpret_cast<int*>(z + L.rowlen),
                                 reinterpret_cast<float*>(z + L.part)},
                         reinterpret_cast<float*>(z + L.logits), reinterpret_cast<unsigned long long*>(z + L.keys),
                         out_tok_dev ? out_tok_dev : reinterpret_cast<int*>(z + L.outtok), nullptr};
        run_step(b, n, false, st_);
        WMI_HIP(hipGetLastError());
    }

    // Adds the stamped cross-attention spans of the last step's nc chains to
    // the WHISPER_K_CROSS_ATTN_STEP totals (joins and waits for the step).
    void read_stamps(int nc) {
        join_chains();
        for (int c = 1; c < nc; ++c) WMI_HIP(hipStreamSynchronize(cst_[c]));
        WMI_HIP(hipStreamSynchronize(st_));
        std::vector<unsigned long long> h((size_t)nc * Ld_ * 2);
        WMI_HIP(hipMemcpy(h.data(), stamps_, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
        Prof& pr = prof_[WHISPER_K_CROSS_ATTN_STEP];
        for (size_t i = 0; i + 1 < h.size(); i += 2) {
            if (h[i + 1] < h[i]) continue;  // a launch without rows
            pr.total_ms += (double)(h[i + 1] - h[i]) / wall_khz_;
            pr.launches += 1;
        }
    }

    // Raises the device-side decode error flag (a row or frame without an
    // admissible token) as an error of the call that synchronised; clears it.
    void check_decode_error() {
        int e = 0;
        WMI_HIP(hipMemcpy(&e, dec_err_, sizeof(int), hipMemcpyDeviceToHost));
        if (e) {
            WMI_HIP(hipMemset(dec_err_, 0, sizeof(int)));
            throw DeviceError(ctc_ ? "CTC head: a frame had no finite logit; the blank was recorded for it"
                                   : "decode step: a row had no admissible token (non-finite logits); token 0 was recorded");
        }
    }

    // Prompt prefill of one encoder pass (prefill_ on): every seated slot's
    // positions 0 .. n_prompt - 2 run through the decoder layers as rows of
    // their own (no output head), writing the self-attention caches. Rows
    // are ordered by position, so a chunk of PF_ROWS rows never needs a
    // position of a later chunk; within a chunk, each layer appends all keys
    // and values before its attention reads them.
    void prefill_pass(const SegmentDesc* segs, int nb, const int* slots) {
        std::vector<int> rows;  // PF list block, then the position block
        int maxp = 0;
        for (int i = 0; i < nb; ++i) maxp = std::max(maxp, segs[i].n_prompt - 1);
        std::vector<int> rl, rp;
        for (int p = 0; p < maxp; ++p)
            for (int i = 0; i < nb; ++i)
                if (p < segs[i].n_prompt - 1) { rl.push_back(slots[i]); rp.push_back(p); }
        const int R = (int)rl.size();
        if (R == 0) return;
        rows.resize(2 * (size_t)pf_cap_);
        for (int c0 = 0; c0 < R; c0 += pf_cap_) {
            const int n = std::min(pf_cap_, R - c0);
            std::copy(rl.begin() + c0, rl.begin() + c0 + n, rows.begin());
            std::copy(rp.begin() + c0, rp.begin() + c0 + n, rows.begin() + pf_cap_);
            upload(3, pf_list_, rows.data(), rows.size() * sizeof(int));
            const RowBufs b{pf_list_, pf_list_ + pf_cap_, pf_dx_, pf_dz_, pf_dq_, pf_datt_, pf_dh_, pf_rowlen_,
                            pf_part_};
            decoder_layers(b, n, st_);
        }
    }

    // Self-attention output projection (x += W_o att + b_o) and the
    // cross-attention queries from LN2(x). bf16 model: the output projection
    // adds the residual itself (no split-K) and the query projection
    // normalises its own input rows, one kernel fewer than the split-K
    // partials + residual/LN kernel + projection of the fp32 model.
    void self_out_cross_q(const DecLayerW<T>& L, int n, const T* datt, T* dq, float* dx, T* dz, float* pbuf,
                          hipStream_t s) {
        const int d = d_;
        if constexpr (std::is_same<T, bf16>::value) {
            if (fused_ln_) {
                skinny_resid(L.Wo, d, datt, n, d, L.bo, dx, s);
                skinny_ln(L.Wcq, d, dx, n, d, L.ln2g, L.ln2b, EpiQ<T>{L.cbq, dq, d}, s);
                return;
            }
        }
        proj_resid(L.Wo, datt, n, d, split_k(d), L.bo, L.ln2g, L.ln2b, pbuf, dx, dz, s);
        proj(L.Wcq, d, dz, n, d, 1, EpiQ<T>{L.cbq, dq, d}, s);
    }

    void read_tokens(int slot, int count, int32_t* dst) override {
        join_chains();
        WMI_HIP(hipSetDevice(dev_));
        if (count <= 0) return;
        WMI_HIP(hipMemcpyAsync(dst, gen_ + (size_t)slot * 448, count * sizeof(int), hipMemcpyDeviceToHost, st_));
        WMI_HIP(hipStreamSynchronize(st_));
    }

    void read_tokens_async(int slot, int count, int32_t* dst) override {
        join_chains();
        queue_read(gen_ + (size_t)slot * 448, count, dst);
    }
    void read_stop_async(int slot, int32_t* dst) override {
        join_chains();
        queue_read(stop_at_ + slot, 1, dst);
    }

    // Queues a copy of count ints from device memory into the pinned area,
    // delivered to dst by finish_reads().
    void queue_read(const int* src, int count, int32_t* dst) {
        if (count <= 0) return;
        if (tokpin_used_ + count > tokpin_cap_) {
            finish_reads();
            if ((size_t)count > tokpin_cap_) {
                if (tokpin_) WMI_HIP(hipHostFree(tokpin_));
                tokpin_ = nullptr;
                tokpin_cap_ = std::max<size_t>(count, 1 << 16);
                WMI_HIP(hipHostMalloc(reinterpret_cast<void**>(&tokpin_), tokpin_cap_ * sizeof(int)));
            }
        }
        WMI_HIP(hipMemcpyAsync(tokpin_ + tokpin_used_, src, count * sizeof(int), hipMemcpyDeviceToHost, st_));
        pending_.push_back({tokpin_used_, count, dst});
        tokpin_used_ += count;
    }

    void finish_reads() override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        for (auto& r : pending_) memcpy(r.dst, tokpin_ + r.off, r.count * sizeof(int));
        pending_.clear();
        tokpin_used_ = 0;
        check_decode_error();
    }

    // -------------------------------------------------------------- decoding options
    void set_decoding(int eot, const int* never, int n_never, const int* first, int n_first) override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        const size_t words = (size_t)V_ / 32 + 1;
        std::vector<unsigned> a(words, 0u), b(words, 0u);
        for (int i = 0; i < n_never; ++i) a[never[i] >> 5] |= 1u << (never[i] & 31);
        for (int i = 0; i < n_first; ++i) b[first[i] >> 5] |= 1u << (first[i] & 31);
        WMI_HIP(hipMemcpy(never_mask_, a.data(), words * 4, hipMemcpyHostToDevice));
        WMI_HIP(hipMemcpy(first_mask_, b.data(), words * 4, hipMemcpyHostToDevice));
        use_never_ = n_never > 0;
        use_first_ = n_first > 0;
        eot_ = eot;
        // the options are launch arguments of the captured steps
        for (auto* m : {&step_graphs_, &stamped_graphs_}) {
            for (auto& g : *m)
                for (auto ge : g.second)
                    if (ge) WMI_HIP(hipGraphExecDestroy(ge));
            m->clear();
        }
    }

    // Snapshot of every slot's stop_at after the work queued so far; poll
    // returns the snapshot taken before the latest one (its copy has long
    // completed when the caller keeps one step ahead), or null.
    void stop_snapshot() override {
        join_chains();
        const int b = (int)(snapshots_ & 1);
        if (!stop_pin_[b]) {
            WMI_HIP(hipHostMalloc(reinterpret_cast<void**>(&stop_pin_[b]), (size_t)S_ * sizeof(int)));
            WMI_HIP(hipEventCreateWithFlags(&stop_ev_[b], hipEventDisableTiming));
        }
        WMI_HIP(hipMemcpyAsync(stop_pin_[b], stop_at_, (size_t)S_ * sizeof(int), hipMemcpyDeviceToHost, st_));
        WMI_HIP(hipEventRecord(stop_ev_[b], st_));
        ++snapshots_;
    }
    const int* stop_poll() override {
        if (snapshots_ < 2) return nullptr;
        const int b = (int)((snapshots_ - 2) & 1);
        WMI_HIP(hipEventSynchronize(stop_ev_[b]));
        return stop_pin_[b];
    }
    void stop_reset() override { snapshots_ = 0; }

    // -------------------------------------------------------------- debug
    void debug_copy(int tensor, int index, void* dst, size_t bytes) override {
        join_chains();
        WMI_HIP(hipSetDevice(dev_));
        WMI_HIP(hipStreamSynchronize(st_));
        float* out = static_cast<float*>(dst);
        if (tensor == WHISPER_T_MEL) {
            need(bytes, (size_t)nm_ * 3000 * 4, index < last_nb_);
            std::vector<float> h((size_t)3000 * nm_);
            WMI_HIP(hipMemcpy(h.data(), logmel_ + (size_t)index * 3000 * nm_, h.size() * 4, hipMemcpyDeviceToHost));
            for (int f = 0; f < 3000; ++f)
                for (int c = 0; c < nm_; ++c) out[(size_t)c * 3000 + f] = h[(size_t)f * nm_ + c];
        } else if (tensor == WHISPER_T_ENC_OUT) {
            need(bytes, (size_t)N_CTX * d_ * 4, index < last_nb_);
            std::vector<T> h((size_t)N_CTX * d_);
            WMI_HIP(hipMemcpy(h.data(), zb_ + (size_t)index * N_CTX * d_, h.size() * sizeof(T), hipMemcpyDeviceToHost));
            for (size_t i = 0; i < h.size(); ++i) out[i] = HostElem<T>::to_f(h.data(), i);
        } else if (tensor == WHISPER_T_CROSS_K || tensor == WHISPER_T_CROSS_V) {
            need(bytes, (size_t)Ld_ * H_ * N_CTX * 64 * 4, index < S_);
            std::vector<T> h((size_t)H_ * 64 * TC);
            for (int l = 0; l < Ld_; ++l) {
                const size_t base = (((size_t)l * S_ + index) * H_) * 64 * TC;
                WMI_HIP(hipMemcpy(h.data(), (tensor == WHISPER_T_CROSS_K ? ktc_ : vc_) + base, h.size() * sizeof(T),
                                  hipMemcpyDeviceToHost));
                for (int hh = 0; hh < H_; ++hh)
                    for (int t = 0; t < N_CTX; ++t)
                        for (int j = 0; j < 64; ++j) {
                            const size_t src = tensor == WHISPER_T_CROSS_K ? ((size_t)hh * 64 + j) * TC + t
                                                                          : ((size_t)hh * TC + t) * 64 + j;
                            out[(((size_t)l * H_ + hh) * N_CTX + t) * 64 + j] = HostElem<T>::to_f(h.data(), src);
                        }
            }
        } else if (tensor == WHISPER_T_CTC_LOGITS && ctc_) {
            need(bytes, (size_t)N_CTX * V_ * 4, index < last_nb_);
            WMI_HIP(hipMemcpy(out, ctc_logits_ + (size_t)index * N_CTX * V_, bytes, hipMemcpyDeviceToHost));
        } else if (tensor == WHISPER_T_CTC_IDS && ctc_) {
            need(bytes, (size_t)N_CTX * 4, index < last_nb_);
            WMI_HIP(hipMemcpy(dst, ctc_ids_ + (size_t)index * N_CTX, bytes, hipMemcpyDeviceToHost));
        } else {
            throw ArgError(WHISPER_E_INVAL, "unknown debug tensor");
        }
    }

    // -------------------------------------------------------------- completion marks
    void mark_reset() override {
        join_chains();
        for (auto e : marks_) event_pool_.push_back(e);
        marks_.clear();
        if (!mark_start_) mark_start_ = get_event();
        WMI_HIP(hipEventRecord(mark_start_, st_));
    }
    int mark() override {
        join_chains();
        hipEvent_t e = get_event();
        WMI_HIP(hipEventRecord(e, st_));
        marks_.push_back(e);
        return (int)marks_.size() - 1;
    }
    std::vector<double> mark_times_us() override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        if (ctc_st_) WMI_HIP(hipStreamSynchronize(ctc_st_));
        std::vector<double> t(marks_.size());
        for (size_t i = 0; i < marks_.size(); ++i) {
            float ms = 0.f;
            WMI_HIP(hipEventElapsedTime(&ms, mark_start_, marks_[i]));
            t[i] = 1e3 * ms;
        }
        return t;
    }

    // -------------------------------------------------------------- profiling
    void profile_enable(int k, bool on) override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        recycle(k);
        prof_[k].on = on;
        prof_[k].total_ms = 0.0;
        prof_[k].launches = 0;
    }
    int encode_ctc(const SegmentDesc* segs, int n, int* mark_out) override {
        join_chains();
        WMI_HIP(hipSetDevice(dev_));
        if (!ctc_) throw ArgError(WHISPER_E_STATE, "not a CTC model");
        if (n < 1 || n > EB_) throw ArgError(WHISPER_E_INVAL, "encode_ctc: 1..max_encode_batch segments");
        const std::vector<int> none(n, 0);
        encode_pass(segs, n, none.data());
        WMI_HIP(hipGetLastError());
        const int ticket = ctc_ticket_++;
        if (mark_out) {  // completion: after the batch's decoding, on the stream that ran it
            hipEvent_t e = get_event();
            WMI_HIP(hipEventRecord(e, P_.ctc_beam >= 2 ? ctc_st_ : st_));
            marks_.push_back(e);
            *mark_out = (int)marks_.size() - 1;
        }
        return ticket;
    }

    void read_ctc(int ticket, int n, int32_t* tokens, int32_t* counts) override {
        join_chains();
        WMI_HIP(hipSetDevice(dev_));
        if (!ctc_ || n < 1 || n > EB_ || ticket < 0 || ticket < ctc_ticket_ - 2 || ticket >= ctc_ticket_)
            throw ArgError(WHISPER_E_INVAL, "read_ctc: one of the last two batches of a CTC model, 1..max_encode_batch entries");
        const int q = ticket & 1;
        WMI_HIP(hipEventSynchronize(ctc_done_[q]));
        WMI_HIP(hipMemcpy(counts, ctc_cnt_[q], n * sizeof(int), hipMemcpyDeviceToHost));
        WMI_HIP(hipMemcpy(tokens, ctc_tok_[q], (size_t)n * N_CTX * sizeof(int), hipMemcpyDeviceToHost));
        check_decode_error();
    }

    double time_cross_attn(int n, int reps) override {
        join_chains();
        WMI_HIP(hipSetDevice(dev_));
        if (n < 1 || n > S_ || reps < 1) throw ArgError(WHISPER_E_INVAL, "time_cross_attn: n in 1..max_slots, reps >= 1");
        std::vector<int> rows(n);
        for (int i = 0; i < n; ++i) rows[i] = i;
        list_host_ = rows;
        upload(0, list_, rows.data(), n * sizeof(int));
        hipEvent_t e0, e1;
        WMI_HIP(hipEventCreate(&e0));
        WMI_HIP(hipEventCreate(&e1));
        WMI_HIP(hipEventRecord(e0, st_));
        for (int i = 0; i < reps; ++i) {
            const long long sl = (long long)(i % Ld_) * S_ * H_ * 64;
            DecAttnArgs ca{dq_, ktc_ + sl * TC, vc_ + sl * TC, datt_, list_, nullptr, TC, H_, d_};
            hipLaunchKernelGGL(cross_attn_kernel<T>, dim3(H_, n), dim3(64 * CW), 0, st_, ca);
        }
        WMI_HIP(hipEventRecord(e1, st_));
        WMI_HIP(hipEventSynchronize(e1));
        float ms = 0.f;
        const hipError_t e = hipEventElapsedTime(&ms, e0, e1);
        (void)hipEventDestroy(e0);
        (void)hipEventDestroy(e1);
        WMI_HIP(e);
        return 1000.0 * ms / reps;
    }

    void profile_read(int k, double* ms, int64_t* launches) override {
        join_chains();
        WMI_HIP(hipStreamSynchronize(st_));
        recycle(k);
        *ms = prof_[k].total_ms;
        *launches = prof_[k].launches;
    }

   private:
    struct Prof {
        bool on = false;
        hipEvent_t open = nullptr;
        std::vector<std::pair<hipEvent_t, hipEvent_t>> used;
        double total_ms = 0.0;
        int64_t launches = 0;
    };
    struct Stage {
        void* host = nullptr;
        size_t cap = 0;
        hipEvent_t ev = nullptr;
    };
    struct PendingRead {
        size_t off;
        int count;
        int32_t* dst;
    };

    whisper_params P_;
    int dev_;
    int d_, H_, Le_, Ld_, V_, nm_, S_, EB_;
    hipStream_t own_stream_ = nullptr, st_ = nullptr;
    std::vector<void*> allocs_;

    unsigned char* scratch_ = nullptr;  // device address of this device's scratch array
    // weights
    T *W1r_, *W2r_, *tok_emb_, *pos_emb_, *WcK_, *WcV_;
    float *cb1_, *cb2_, *lnpg_, *lnpb_, *lnfg_, *lnfb_, *bcV_;
    std::vector<EncLayerW<T>> enc_;
    std::vector<DecLayerW<T>> dec_;
    float *basis_, *melfb_, *pe_;
    // encoder workspace
    float *stage_audio_, *xpad_, *power_, *logmel_, *melmax_, *x_;
    SegSrc* segsrc_;
    int *nvalid_, *slot_of_, *seat_np_, *seat_prompts_;
    T *ypad_, *h1_, *zb_, *qh_, *kh_, *vt_, *ob_, *hb_;
    int last_nb_ = 0;
    // decoder state and workspace
    int *seq_, *gen_, *pos_, *npr_, *list_, *forced_, *outtok_, *rowlen_, *stop_at_;
    // decoding options: logit filter masks, end-of-text token (-1: none)
    unsigned *never_mask_, *first_mask_;
    bool use_never_ = false, use_first_ = false;
    int eot_ = -1;
    int* stop_pin_[2] = {nullptr, nullptr};
    hipEvent_t stop_ev_[2] = {nullptr, nullptr};
    int64_t snapshots_ = 0;
    T *kts_, *vs_, *ktc_, *vc_, *dz_, *dq_, *datt_, *dh_;
    float *dx_, *logits_, *gpart_;
    unsigned long long* keys_;  // greedy-choice keys [S][nkeys_]
    int nkeys_ = ARGMAX_CHUNKS;
    int* dec_err_;              // set by a decode step that found no admissible token
    std::vector<int> list_host_;
    bool graphs_ = true, split_ = true, fused_ln_ = true;
    bool free_run_ = true, chains_apart_ = false;
    static constexpr int KSMAX = 8;  // most split-K partials of a decode projection
    int fc2_split_ = 8;  // split-K of fc2 (K = 4d) where 4d / 32 is a multiple of 8
    int apart_nc_ = 0;
    // prompt prefill: rows per chunk (the skinny projections take up to 128)
    // and the chunk's buffers; the list block is followed by the positions
    bool prefill_ = false;
    int pf_cap_ = 0;
    int *pf_list_ = nullptr, *pf_rowlen_ = nullptr;
    float *pf_dx_ = nullptr, *pf_part_ = nullptr;
    T *pf_dz_ = nullptr, *pf_dq_ = nullptr, *pf_datt_ = nullptr, *pf_dh_ = nullptr;
    bool ctc_ = false;  // encoder-only CTC model (no decoder layers)
    T* Wctc_ = nullptr;
    float* bctc_ = nullptr;
    float* ctc_logits_ = nullptr;  // [max_encode_batch * 1500][n_vocab]
    int* ctc_ids_ = nullptr;
    // per ticket parity (two batches in flight): labels and counts; beam
    // search: frame counts, per-frame blank and candidate log-probs,
    // candidate ids, backpointers
    int *ctc_tok_[2] = {}, *ctc_cnt_[2] = {}, *ctc_T_[2] = {};
    float *ctc_lpb_[2] = {}, *ctc_clp_[2] = {};
    int *ctc_cid_[2] = {}, *ctc_bp_[2] = {};
    int ctc_ticket_ = 0;
    hipStream_t ctc_st_ = nullptr;  // beam search of one batch beside the next batch's encoder
    hipEvent_t ctc_head_[2] = {}, ctc_done_[2] = {};
    static constexpr int MAXC = 4;                                  // chains of a step (hardware queues)
    int chains_ = 2;
    std::map<int, std::array<hipGraphExec_t, MAXC>> step_graphs_;  // per row count: one graph per chain
    std::map<int, std::array<hipGraphExec_t, MAXC>> stamped_graphs_;  // the same with cross-attention stamps
    bool stamp_on_ = false;                 // launches being made carry cross-attention stamps
    unsigned long long* stamps_ = nullptr;  // [chain][layer][2] stamp slots
    double wall_khz_ = 100000.0;            // real-time counter ticks per millisecond
    hipStream_t cst_[MAXC] = {};                                   // streams of chains 1.. (chain 0: st_)
    static constexpr int ENC_PARTS_MAX = 4;
    hipStream_t es_[ENC_PARTS_MAX - 1] = {};                       // the encoder pass's parts 1..
    hipEvent_t enc_fork_ = nullptr, enc_join_[ENC_PARTS_MAX - 1] = {};
    int enc_parts_ = 2;
    hipEvent_t fork_ev_ = nullptr, join_ev_[MAXC] = {};
    // host staging
    Stage stage_[4];
    int32_t* tokpin_ = nullptr;
    size_t tokpin_cap_ = 0, tokpin_used_ = 0;
    std::vector<PendingRead> pending_;
    Prof prof_[WHISPER_K_COUNT];
    std::vector<hipEvent_t> event_pool_;
    hipEvent_t mark_start_ = nullptr;
    std::vector<hipEvent_t> marks_;

    template <class U>
    U* dalloc(size_t count) {
        void* q = nullptr;
        if (hipMalloc(&q, std::max<size_t>(count, 1) * sizeof(U)) != hipSuccess)
            throw ArgError(WHISPER_E_NOMEM, "device allocation of " + std::to_string(count * sizeof(U)) + " bytes failed");
        allocs_.push_back(q);
        WMI_HIP(hipMemset(q, 0, std::max<size_t>(count, 1) * sizeof(U)));
        return static_cast<U*>(q);
    }
    template <class U>
    U* upload_new(const std::vector<U>& h) {
        U* q = dalloc<U>(h.size());
        WMI_HIP(hipMemcpy(q, h.data(), h.size() * sizeof(U), hipMemcpyHostToDevice));
        return q;
    }

    // Copies host bytes to device memory through pinned staging area `which`
    // (waits for the previous copy from that area first).
    void upload(int which, void* dst, const void* src, size_t bytes) {
        Stage& s = stage_[which];
        if (s.ev) WMI_HIP(hipEventSynchronize(s.ev));
        else WMI_HIP(hipEventCreateWithFlags(&s.ev, hipEventDisableTiming));
        if (bytes > s.cap) {
            if (s.host) WMI_HIP(hipHostFree(s.host));
            s.host = nullptr;
            s.cap = std::max<size_t>(bytes, 4096);
            WMI_HIP(hipHostMalloc(&s.host, s.cap));
        }
        memcpy(s.host, src, bytes);
        WMI_HIP(hipMemcpyAsync(dst, s.host, bytes, hipMemcpyHostToDevice, st_));
        WMI_HIP(hipEventRecord(s.ev, st_));
    }

    hipEvent_t get_event() {
        if (!event_pool_.empty()) { hipEvent_t e = event_pool_.back(); event_pool_.pop_back(); return e; }
        hipEvent_t e;
        WMI_HIP(hipEventCreate(&e));
        return e;
    }
    void prof_begin(int k, hipStream_t s) {
        if (!prof_[k].on) return;
        prof_[k].open = get_event();
        WMI_HIP(hipEventRecord(prof_[k].open, s));
    }
    void prof_end(int k, hipStream_t s) {
        if (!prof_[k].on) return;
        hipEvent_t e = get_event();
        WMI_HIP(hipEventRecord(e, s));
        prof_[k].used.push_back({prof_[k].open, e});
        if (prof_[k].used.size() >= 4096) {  // bound the number of live events
            WMI_HIP(hipStreamSynchronize(st_));
            recycle(k);
        }
    }
    void recycle(int k) {
        for (auto& pr : prof_[k].used) {
            float ms = 0.f;
            WMI_HIP(hipEventElapsedTime(&ms, pr.first, pr.second));
            prof_[k].total_ms += ms;
            prof_[k].launches += 1;
            event_pool_.push_back(pr.first);
            event_pool_.push_back(pr.second);
        }
        prof_[k].used.clear();
    }

    static void need(size_t got, size_t want, bool index_ok) {
        if (!index_ok) throw ArgError(WHISPER_E_INVAL, "debug_copy: index out of range");
        if (got != want)
            throw ArgError(WHISPER_E_BUFFER, "debug_copy: buffer must hold exactly " + std::to_string(want) + " bytes");
    }

    // -------------------------------------------------------------- kernels
    void ln(const float* x, T* y, const float* g, const float* b, int rows, hipStream_t s = nullptr) {
        WMI_SWITCH_E(d_, hipLaunchKernelGGL((layer_norm_kernel<T, E>), dim3((rows + 3) / 4), dim3(256), 0,
                                            s ? s : st_, x, y, g, b, rows));
    }
    // decoder: x += split-K partials + bias, then z = LN(x)
    void resid_ln(int KS, int n, const float* bias, const float* g, const float* b, float* part, float* dx, T* dz,
                  hipStream_t s) {
        if (KS == 8) {
            WMI_SWITCH_E(d_, hipLaunchKernelGGL((resid_ln_kernel<T, E, 8>), dim3(n), dim3(resid_ln_threads<E>()), 0,
                                                s, part, n, bias, dx, dz, g, b));
        } else if (KS == 4) {
            WMI_SWITCH_E(d_, hipLaunchKernelGGL((resid_ln_kernel<T, E, 4>), dim3(n), dim3(resid_ln_threads<E>()), 0,
                                                s, part, n, bias, dx, dz, g, b));
        } else {
            WMI_SWITCH_E(d_, hipLaunchKernelGGL((resid_ln_kernel<T, E, 1>), dim3(n), dim3(resid_ln_threads<E>()), 0,
                                                s, part, n, bias, dx, dz, g, b));
        }
    }
    // log-mel of `frames` power rows on the matrix cores (mel tiles of 16)
    void mel_log(int frames) {
        const dim3 grid((frames + 63) / 64);
        switch ((nm_ + 15) / 16) {
#define WMI_MEL_CASE(MT) \
    case MT: hipLaunchKernelGGL(mel_log_kernel<MT>, grid, dim3(256), 0, st_, melfb_, power_, logmel_, frames, nm_); break;
            WMI_MEL_CASE(1) WMI_MEL_CASE(2) WMI_MEL_CASE(3) WMI_MEL_CASE(4)
            WMI_MEL_CASE(5) WMI_MEL_CASE(6) WMI_MEL_CASE(7) WMI_MEL_CASE(8)
#undef WMI_MEL_CASE
            default: throw ArgError(WHISPER_E_INVAL, "n_mels above 128");
        }
    }

    // split factor of a decode projection with reduction length K
    static int split_k(int K) { return (K / 32) % 4 == 0 ? 4 : 1; }

    template <class Epi>
    void gemm(const T* A, int lda, long long sA, const T* B, int ldb, long long sB, int MA, int MB, int K, int batch,
              const Epi& epi, hipStream_t s = nullptr) {
        if (!s) s = st_;
        if constexpr (std::is_same<T, bf16>::value) gemm_bf16(A, lda, sA, B, ldb, sB, MA, MB, K, batch, epi, s);
        else gemm_simt(A, lda, sA, B, ldb, sB, MA, MB, K, batch, epi, s);
    }

    // Encoder layer l over segments b0 .. b0 + nb - 1 of the pass, on stream
    // s: every buffer is addressed from that segment range, so two ranges
    // can run on two streams at once.
    void encoder_layer(int l, int b0, int nb, hipStream_t s) {
        const EncLayerW<T>& L = enc_[l];
        const int d = d_, M = nb * N_CTX;
        const long long tok = (long long)b0 * N_CTX, head = (long long)b0 * H_ * TQ * 64;
        float* x = x_ + tok * d;
        T* zb = zb_ + tok * d;
        T* qh = qh_ + head;
        T* kh = kh_ + head;
        T* vt = vt_ + head;
        T* ob = ob_ + tok * d;
        T* hb = hb_ + tok * 4 * d;
        ln(x, zb, L.ln1g, L.ln1b, M, s);
        gemm(L.Wqk, d, 0, zb, d, 0, 2 * d, M, d, 1, EpiQK<T>{L.bq, qh, kh, d, H_}, s);
        gemm(zb, d, 0, L.Wv, d, 0, M, d, d, 1, EpiVt<T>{L.bv, vt, H_}, s);
        prof_begin(WHISPER_K_ENC_ATTN, s);
        if constexpr (std::is_same<T, bf16>::value)
            hipLaunchKernelGGL(enc_attn_bf16_kernel, dim3((N_CTX + ea::QB - 1) / ea::QB, nb * H_), dim3(256), 0, s,
                               qh, kh, vt, ob, H_, d);
        else
            hipLaunchKernelGGL(enc_attn_f32_kernel, dim3((N_CTX + 63) / 64, nb * H_), dim3(64), 0, s, qh, kh, vt, ob,
                               H_, d);
        prof_end(WHISPER_K_ENC_ATTN, s);
        gemm(L.Wo, d, 0, ob, d, 0, d, M, d, 1, EpiResid{L.bo, x, d}, s);
        ln(x, zb, L.ln2g, L.ln2b, M, s);
        prof_begin(WHISPER_K_ENC_GEMM, s);
        gemm(L.W1, d, 0, zb, d, 0, 4 * d, M, d, 1, EpiGelu<T>{L.b1, hb, 4 * d}, s);
        prof_end(WHISPER_K_ENC_GEMM, s);
        gemm(L.W2, 4 * d, 0, hb, 4 * d, 0, d, M, 4 * d, 1, EpiResid{L.b2, x, d}, s);
    }

    // decode projection: rows = weight rows (MA), n activation rows of width K
    template <class Epi>
    void proj(const T* W, int MA, const T* X, int n, int K, int KS, const Epi& epi, hipStream_t s) {
        if constexpr (std::is_same<T, bf16>::value) skinny_bf16(W, MA, X, n, K, KS, epi, s);
        else gemm_simt(W, K, K / KS, X, K, K / KS, MA, n, K / KS, KS, epi, s);
    }
    // residual projection: x += W X + bias (split-K partials), then z = LN(x)
    void proj_resid(const T* W, const T* X, int n, int K, int KS, const float* bias, const float* g, const float* b,
                    float* part, float* dx, T* dz, hipStream_t s) {
        proj(W, d_, X, n, K, KS, EpiPartial{part, d_, n}, s);
        resid_ln(KS, n, bias, g, b, part, dx, dz, s);
    }

    void encode_pass(const SegmentDesc* segs, int nb, const int* slots) {
        const int d = d_, M = nb * N_CTX;
        // small per-pass arrays: sources, valid frames, slots, prompts
        std::vector<SegSrc> src(nb);
        // nvalid | slot_of | n_prompt | prompts, each block EB entries long (the
        // device pointers nvalid_, slot_of_, seat_np_, seat_prompts_ use that stride)
        std::vector<int> small((size_t)EB_ * (3 + 448), 0);
        int* nv = small.data();
        int* so = nv + EB_;
        int* npv = so + EB_;
        int* pr = npv + EB_;
        for (int i = 0; i < nb; ++i) {
            const SegmentDesc& s = segs[i];
            if (s.on_device) {
                src[i] = SegSrc{s.audio, s.n_samples, 0};
            } else {
                float* dst = stage_audio_ + (size_t)i * 480000;
                WMI_HIP(hipMemcpyAsync(dst, s.audio, (size_t)s.n_samples * 4, hipMemcpyHostToDevice, st_));
                src[i] = SegSrc{dst, s.n_samples, 0};
            }
            nv[i] = P_.pad_mode == 0 ? 3000 : s.n_samples / 160;
            // decoder models: the slot; CTC models: the encoder frames covering
            // the audio (320 samples each), the frames greedy decoding reads
            so[i] = ctc_ ? std::min(N_CTX, (s.n_samples + 319) / 320) : slots[i];
            npv[i] = s.n_prompt;
            memcpy(pr + (size_t)i * 448, s.prompt, s.n_prompt * sizeof(int));
        }
        upload(2, segsrc_, src.data(), nb * sizeof(SegSrc));
        // the three int arrays and prompts live contiguously behind nvalid_
        WMI_HIP(hipEventSynchronize(stage_[2].ev));
        upload(2, nvalid_, small.data(), small.size() * sizeof(int));
        last_nb_ = nb;

        prof_begin(WHISPER_K_ENC_PASS, st_);
        prof_begin(WHISPER_K_FRONT_END, st_);
        hipLaunchKernelGGL(prep_audio_kernel, dim3((480400 + 255) / 256, nb), dim3(256), 0, st_, segsrc_, xpad_,
                           P_.pad_mode);
        hipLaunchKernelGGL(dft_power_kernel, dim3((3000 + DFT_FB - 1) / DFT_FB, 2, nb), dim3(256), 0, st_, basis_,
                           xpad_, power_);
        mel_log(nb * 3000);
        hipLaunchKernelGGL(mel_max_kernel, dim3(MEL_CHUNKS, nb), dim3(256), 0, st_, logmel_, nvalid_, nm_, melmax_);
        hipLaunchKernelGGL(mel_norm_kernel<T>, dim3(64, nb), dim3(256), 0, st_, logmel_, ypad_, nvalid_, nm_, melmax_);
        prof_end(WHISPER_K_FRONT_END, st_);
        gemm(W1r_, 3 * CP, 0, ypad_, CP, 3002LL * CP, d, 3000, 3 * CP, nb, EpiConv1<T>{cb1_, h1_, d});
        gemm(W2r_, 3 * d, 0, h1_, 2 * d, 3002LL * d, d, N_CTX, 3 * d, nb, EpiConv2{cb2_, pe_, x_, d});
        // The pass in parts of its segments on parallel streams (bf16
        // models): the segments are independent, and the parts' kernels fill
        // each other's partial last rounds and spread the epilogues' memory
        // phases. With the per-kernel encoder timers on, one stream, so each
        // timed launch covers the whole pass.
        const int parts = std::is_same<T, bf16>::value && !prof_[WHISPER_K_ENC_GEMM].on &&
                                  !prof_[WHISPER_K_ENC_ATTN].on
                              ? std::min(enc_parts_, nb)
                              : 1;
        if (parts > 1) {
            WMI_HIP(hipEventRecord(enc_fork_, st_));
            for (int k = 1; k < parts; ++k) WMI_HIP(hipStreamWaitEvent(es_[k - 1], enc_fork_, 0));
            for (int l = 0; l < Le_; ++l)
                for (int k = 0; k < parts; ++k) {
                    const int b0 = nb * k / parts, b1 = nb * (k + 1) / parts;
                    encoder_layer(l, b0, b1 - b0, k == 0 ? st_ : es_[k - 1]);
                }
            for (int k = 1; k < parts; ++k) {
                WMI_HIP(hipEventRecord(enc_join_[k - 1], es_[k - 1]));
                WMI_HIP(hipStreamWaitEvent(st_, enc_join_[k - 1], 0));
            }
        } else {
            for (int l = 0; l < Le_; ++l) encoder_layer(l, 0, nb, st_);
        }
        ln(x_, zb_, lnpg_, lnpb_, M);
        if (ctc_) {  // CTC head, per-frame argmax, then decoding into the ticket's buffers
            const int q = ctc_ticket_ & 1;
            gemm(Wctc_, d, 0, zb_, d, 0, V_, M, d, 1, EpiCTC{bctc_, ctc_logits_, V_});
            hipLaunchKernelGGL(ctc_argmax_kernel, dim3((M + 3) / 4), dim3(256), 0, st_, ctc_logits_, V_, M, ctc_ids_,
                               dec_err_);
            // the batch before last used these buffers: its search must be done
            WMI_HIP(hipStreamWaitEvent(st_, ctc_done_[q], 0));
            if (P_.ctc_beam >= 2) {
                // candidates on this stream; the search itself on the side
                // stream, where it overlaps the next batch's encoder
                hipLaunchKernelGGL(ctc_frame_topk_kernel, dim3((M + 3) / 4), dim3(256), 0, st_, ctc_logits_, V_, M,
                                   P_.ctc_beam, ctc_lpb_[q], ctc_cid_[q], ctc_clp_[q]);
                WMI_HIP(hipMemcpyAsync(ctc_T_[q], slot_of_, nb * sizeof(int), hipMemcpyDeviceToDevice, st_));
                WMI_HIP(hipEventRecord(ctc_head_[q], st_));
                WMI_HIP(hipStreamWaitEvent(ctc_st_, ctc_head_[q], 0));
                hipLaunchKernelGGL(ctc_beam_kernel, dim3(nb), dim3(64), 0, ctc_st_, ctc_lpb_[q], ctc_cid_[q],
                                   ctc_clp_[q], ctc_T_[q], P_.ctc_beam, P_.ctc_beam, ctc_bp_[q], ctc_tok_[q],
                                   ctc_cnt_[q]);
                WMI_HIP(hipEventRecord(ctc_done_[q], ctc_st_));
            } else {
                hipLaunchKernelGGL(ctc_collapse_kernel, dim3(nb), dim3(1024), 0, st_, ctc_ids_, slot_of_, ctc_tok_[q],
                                   ctc_cnt_[q]);
                WMI_HIP(hipEventRecord(ctc_done_[q], st_));
            }
            prof_end(WHISPER_K_ENC_PASS, st_);
            return;
        }
        gemm(zb_, d, 0, WcK_, d, 0, M, Ld_ * d, d, 1, EpiCrossK<T>{ktc_, slot_of_, d, H_, S_, 1.0f / d});
        gemm(WcV_, d, 0, zb_, d, 0, Ld_ * d, M, d, 1, EpiCrossV<T>{bcV_, vc_, slot_of_, d, H_, S_, 1.0f / d});
        hipLaunchKernelGGL(seat_kernel, dim3(nb), dim3(256), 0, st_, slot_of_, seat_np_, seat_prompts_, seq_, pos_, npr_,
                           stop_at_, prefill_ ? 1 : 0);
        prof_end(WHISPER_K_ENC_PASS, st_);
        if (prefill_) prefill_pass(segs, nb, slots);
    }

    // -------------------------------------------------------------- setup
    void load_weights(const void* blob, size_t bytes) {
        std::map<std::string, std::pair<size_t, long long>> offs;
        const size_t want = blob_size(P_, &offs);
        if (bytes != want)
            throw ArgError(WHISPER_E_FORMAT, "weight blob has " + std::to_string(bytes) + " bytes, layout needs " +
                                                 std::to_string(want));
        const char* base = static_cast<const char*>(blob);
        auto raw = [&](const std::string& name) -> const T* {
            return reinterpret_cast<const T*>(base + offs.at(name).first);
        };
        auto count = [&](const std::string& name) { return (size_t)offs.at(name).second; };
        auto mat = [&](const std::string& name) -> T* {
            T* q = dalloc<T>(count(name));
            WMI_HIP(hipMemcpy(q, raw(name), count(name) * sizeof(T), hipMemcpyHostToDevice));
            return q;
        };
        auto vecf = [&](const std::string& name) -> float* {
            std::vector<float> h(count(name));
            for (size_t i = 0; i < h.size(); ++i) h[i] = HostElem<T>::to_f(raw(name), i);
            return upload_new(h);
        };
        auto cat = [&](const std::vector<std::string>& names) -> T* {
            size_t tot = 0;
            for (auto& nme : names) tot += count(nme);
            T* q = dalloc<T>(tot);
            size_t o = 0;
            for (auto& nme : names) {
                WMI_HIP(hipMemcpy(q + o, raw(nme), count(nme) * sizeof(T), hipMemcpyHostToDevice));
                o += count(nme);
            }
            return q;
        };
        // Decoder projection matrices with K columns (rows of the named tensors
        // stacked) in the decoder layout: bf16 fragment-major with the rows
        // padded with zeros to a multiple of 32, fp32 row-major.
        auto dec_mat = [&](const std::vector<std::string>& names, int K) -> T* {
            if constexpr (!std::is_same<T, bf16>::value) {
                return cat(names);
            } else {
                size_t rows = 0;
                for (auto& nme : names) rows += count(nme) / K;
                std::vector<T> h((rows + 31) / 32 * 32 * K);
                memset(h.data(), 0, h.size() * sizeof(T));
                size_t r0 = 0;
                for (auto& nme : names) {
                    const T* src = raw(nme);
                    const size_t nr = count(nme) / K;
                    for (size_t r = 0; r < nr; ++r)
                        for (int k = 0; k < K; k += 8)
                            memcpy(&h[frag_off(r0 + r, k, K)], src + r * K + k, 8 * sizeof(T));
                    r0 += nr;
                }
                return upload_new(h);
            }
        };
        const int d = d_;
        {  // conv kernels to [out][tap][in] (input channels of conv1 padded to CP)
            std::vector<T> w1((size_t)d * 3 * CP);
            memset(w1.data(), 0, w1.size() * sizeof(T));
            const T* s1 = raw("enc.conv1.w");
            for (int o = 0; o < d; ++o)
                for (int c = 0; c < nm_; ++c)
                    for (int t = 0; t < 3; ++t) w1[(size_t)o * 3 * CP + t * CP + c] = s1[((size_t)o * nm_ + c) * 3 + t];
            W1r_ = upload_new(w1);
            std::vector<T> w2((size_t)d * 3 * d);
            const T* s2 = raw("enc.conv2.w");
            for (int o = 0; o < d; ++o)
                for (int c = 0; c < d; ++c)
                    for (int t = 0; t < 3; ++t) w2[(size_t)o * 3 * d + t * d + c] = s2[((size_t)o * d + c) * 3 + t];
            W2r_ = upload_new(w2);
        }
        cb1_ = vecf("enc.conv1.b");
        cb2_ = vecf("enc.conv2.b");
        for (int i = 0; i < Le_; ++i) {
            const std::string p = "enc." + std::to_string(i);
            EncLayerW<T> L;
            L.ln1g = vecf(p + ".attn_ln.g"); L.ln1b = vecf(p + ".attn_ln.b");
            L.Wqk = cat({p + ".attn.q.w", p + ".attn.k.w"});
            L.bq = vecf(p + ".attn.q.b");
            L.Wv = mat(p + ".attn.v.w"); L.bv = vecf(p + ".attn.v.b");
            L.Wo = mat(p + ".attn.o.w"); L.bo = vecf(p + ".attn.o.b");
            L.ln2g = vecf(p + ".mlp_ln.g"); L.ln2b = vecf(p + ".mlp_ln.b");
            L.W1 = mat(p + ".mlp.fc1.w"); L.b1 = vecf(p + ".mlp.fc1.b");
            L.W2 = mat(p + ".mlp.fc2.w"); L.b2 = vecf(p + ".mlp.fc2.b");
            enc_.push_back(L);
        }
        lnpg_ = vecf("enc.ln_post.g");
        lnpb_ = vecf("enc.ln_post.b");
        basis_ = upload_new(dft_basis());
        {  // k-major [DFT_PS][mel tiles x 16], zero beyond bin 200 and mel nm_ - 1
            const int mp = (nm_ + 15) / 16 * 16;
            const std::vector<float> fb = mel_bank(nm_);
            std::vector<float> t((size_t)DFT_PS * mp, 0.f);
            for (int m = 0; m < nm_; ++m)
                for (int k = 0; k < 201; ++k) t[(size_t)k * mp + m] = fb[(size_t)m * 201 + k];
            melfb_ = upload_new(t);
        }
        pe_ = upload_new(sinusoids(N_CTX, d));
        if (ctc_) {
            Wctc_ = mat("ctc.w");
            bctc_ = vecf("ctc.b");
            return;
        }
        tok_emb_ = dec_mat({"dec.tok_emb"}, d);
        pos_emb_ = mat("dec.pos_emb");
        std::vector<std::string> ck, cv;
        std::vector<float> bcv;
        for (int i = 0; i < Ld_; ++i) {
            const std::string p = "dec." + std::to_string(i);
            DecLayerW<T> L;
            L.ln1g = vecf(p + ".attn_ln.g"); L.ln1b = vecf(p + ".attn_ln.b");
            L.Wqkv = dec_mat({p + ".attn.q.w", p + ".attn.k.w", p + ".attn.v.w"}, d);
            L.bq = vecf(p + ".attn.q.b"); L.bv = vecf(p + ".attn.v.b");
            L.Wo = dec_mat({p + ".attn.o.w"}, d); L.bo = vecf(p + ".attn.o.b");
            L.ln2g = vecf(p + ".cross_ln.g"); L.ln2b = vecf(p + ".cross_ln.b");
            L.Wcq = dec_mat({p + ".cross.q.w"}, d); L.cbq = vecf(p + ".cross.q.b");
            L.Wco = dec_mat({p + ".cross.o.w"}, d); L.cbo = vecf(p + ".cross.o.b");
            L.ln3g = vecf(p + ".mlp_ln.g"); L.ln3b = vecf(p + ".mlp_ln.b");
            L.W1 = dec_mat({p + ".mlp.fc1.w"}, d); L.b1 = vecf(p + ".mlp.fc1.b");
            L.W2 = dec_mat({p + ".mlp.fc2.w"}, 4 * d); L.b2 = vecf(p + ".mlp.fc2.b");
            dec_.push_back(L);
            ck.push_back(p + ".cross.k.w");
            cv.push_back(p + ".cross.v.w");
            const T* b = raw(p + ".cross.v.b");
            for (int j = 0; j < d; ++j) bcv.push_back(HostElem<T>::to_f(b, j));
        }
        WcK_ = cat(ck);
        WcV_ = cat(cv);
        bcV_ = upload_new(bcv);
        lnfg_ = vecf("dec.ln.g");
        lnfb_ = vecf("dec.ln.b");
    }

    void alloc_state() {
        const size_t d = d_, H = H_, EB = EB_, S = S_, Ld = Ld_;
        stage_audio_ = dalloc<float>(EB * 480000);
        segsrc_ = dalloc<SegSrc>(EB);
        nvalid_ = dalloc<int>(EB * (3 + 448));
        slot_of_ = nvalid_ + EB;
        seat_np_ = slot_of_ + EB;
        seat_prompts_ = seat_np_ + EB;
        xpad_ = dalloc<float>(EB * 480400);
        power_ = dalloc<float>(EB * 3000 * DFT_PS);
        logmel_ = dalloc<float>(EB * 3000 * nm_);
        melmax_ = dalloc<float>(EB * MEL_CHUNKS);
        ypad_ = dalloc<T>(EB * 3002 * CP);
        h1_ = dalloc<T>(EB * 3002 * d);
        x_ = dalloc<float>(EB * N_CTX * d);
        zb_ = dalloc<T>(EB * N_CTX * d);
        qh_ = dalloc<T>(EB * H * TQ * 64);
        kh_ = dalloc<T>(EB * H * TQ * 64);
        vt_ = dalloc<T>(EB * H * 64 * TQ);
        ob_ = dalloc<T>(EB * N_CTX * d);
        hb_ = dalloc<T>(EB * N_CTX * 4 * d);
        seq_ = dalloc<int>(S * 448);
        gen_ = dalloc<int>(S * 448);
        pos_ = dalloc<int>(S);
        npr_ = dalloc<int>(S);
        list_ = dalloc<int>(S);
        forced_ = dalloc<int>(S);
        outtok_ = dalloc<int>(S);
        rowlen_ = dalloc<int>(S);
        stop_at_ = dalloc<int>(S);
        never_mask_ = dalloc<unsigned>((size_t)V_ / 32 + 1);
        first_mask_ = dalloc<unsigned>((size_t)V_ / 32 + 1);
        kts_ = dalloc<T>(Ld * S * H * 64 * TS);
        vs_ = dalloc<T>(Ld * S * H * TS * 64);
        ktc_ = dalloc<T>(Ld * S * H * 64 * TC);
        vc_ = dalloc<T>(Ld * S * H * TC * 64);
        // activations multiplied by projections: whole 16-row tiles (fragment-major in bf16)
        const size_t S16 = (S + 15) / 16 * 16;
        dx_ = dalloc<float>(S * d);
        dz_ = dalloc<T>(S16 * d);
        dq_ = dalloc<T>(S * d);
        datt_ = dalloc<T>(S16 * d);
        dh_ = dalloc<T>(S16 * 4 * d);
        logits_ = dalloc<float>(S * (size_t)V_);
        gpart_ = dalloc<float>((size_t)MAXC * KSMAX * S * d);  // split-K partials [chain][KS][rows][d]
        stamps_ = dalloc<unsigned long long>((size_t)MAXC * std::max(Ld_, 1) * 2);
        {
            int khz = 0;
            if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev_) == hipSuccess && khz > 0)
                wall_khz_ = khz;
        }
        nkeys_ = std::max(ARGMAX_CHUNKS, (V_ + 31) / 32);
        keys_ = dalloc<unsigned long long>(S * (size_t)nkeys_);
        dec_err_ = dalloc<int>(1);
        if (prefill_) {
            pf_cap_ = 128;
            pf_list_ = dalloc<int>(2 * pf_cap_);
            pf_rowlen_ = dalloc<int>(pf_cap_);
            pf_dx_ = dalloc<float>((size_t)pf_cap_ * d);
            pf_dz_ = dalloc<T>((size_t)pf_cap_ * d);
            pf_dq_ = dalloc<T>((size_t)pf_cap_ * d);
            pf_datt_ = dalloc<T>((size_t)pf_cap_ * d);
            pf_dh_ = dalloc<T>((size_t)pf_cap_ * 4 * d);
            pf_part_ = dalloc<float>((size_t)KSMAX * pf_cap_ * d);
        }
        if (ctc_) {
            ctc_logits_ = dalloc<float>(EB * N_CTX * (size_t)V_);
            ctc_ids_ = dalloc<int>(EB * N_CTX);
            WMI_HIP(hipStreamCreateWithFlags(&ctc_st_, hipStreamNonBlocking));
            for (int q = 0; q < 2; ++q) {  // two batches in flight: buffers by ticket parity
                ctc_tok_[q] = dalloc<int>(EB * N_CTX);
                ctc_cnt_[q] = dalloc<int>(EB);
                WMI_HIP(hipEventCreateWithFlags(&ctc_head_[q], hipEventDisableTiming));
                WMI_HIP(hipEventCreateWithFlags(&ctc_done_[q], hipEventDisableTiming));
                WMI_HIP(hipEventRecord(ctc_done_[q], st_));
                if (P_.ctc_beam >= 2) {
                    ctc_T_[q] = dalloc<int>(EB);
                    ctc_lpb_[q] = dalloc<float>(EB * N_CTX);
                    ctc_cid_[q] = dalloc<int>(EB * N_CTX * cb::KMAX);
                    ctc_clp_[q] = dalloc<float>(EB * N_CTX * cb::KMAX);
                    ctc_bp_[q] = dalloc<int>(EB * N_CTX * cb::KMAX);
                }
            }
        }
    }
};

// Host run of the greedy choice's key arithmetic (amax_key, key_token): the
// admissible ids of each row (bit clear in `excluded`, [V / 32 + 1] words,
// or null) become keys, the largest key per row is decoded.
void greedy_keys_host(const float* logits, int rows, int V, const unsigned* excluded, int* tokens, int* bad) {
    for (int r = 0; r < rows; ++r) {
        unsigned long long k = 0;
        for (int i = 0; i < V; ++i) {
            if (excluded && ((excluded[i >> 5] >> (i & 31)) & 1u)) continue;
            const unsigned long long c = amax_key(logits[(size_t)r * V + i], i);
            k = c > k ? c : k;
        }
        bad[r] = 0;
        tokens[r] = key_token(k, &bad[r]);
    }
}

std::unique_ptr<Engine> make_engine(const whisper_params& p, const void* blob, size_t bytes, int device) {
    if (p.dtype == WHISPER_DTYPE_BF16) return std::unique_ptr<Engine>(new EngineT<bf16>(p, blob, bytes, device));
    return std::unique_ptr<Engine>(new EngineT<float>(p, blob, bytes, device));
}

}  // namespace wmi
