// Context, validation, planning and the layer-by-layer launch sequence behind
// the kvr_* C interface.
//
// One pass runs the decoder over a set of rows (positions of one or more
// documents) against those documents' caches: embedding gather, then per layer
// RMSNorm -> QKV projection -> rotary embedding + scatter of the fresh K/V into
// the cache -> causal attention over the cache -> output projection (+
// residual) -> RMSNorm -> gate/up projection with SwiGLU -> down projection (+
// residual), and a final RMSNorm into the caller's output rows.  Repair is one
// pass over P = S u A (paper Section 3, "The repair interface"); prefill is a
// pass (or consecutive chunks of passes) over all positions.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/kvr.h"
#include "common.h"

using namespace kvr;

namespace kvr {

static thread_local std::string g_error;
void set_global_error(const char *msg) { g_error = msg; }

LaunchTimer &launch_timer() {
    static thread_local LaunchTimer t;
    return t;
}

// The host tables of one pass.  A context keeps one set, reserved to its
// capacities when it is created, so that planning a pass allocates nothing.
struct Tables {
    struct Block { int doc, row0, nrows, kmax; };  // attention row block (planner)
    std::vector<RowInfo> rows;
    std::vector<DocInfo> docs;
    std::vector<AttnItem> items;
    std::vector<CombineItem> comb;
    std::vector<Block> blocks;
    int att_mt = 1;  // 16-row tiles per attention item (rows of a row block / 16)
    void clear() {
        rows.clear(); docs.clear(); items.clear(); comb.clear(); blocks.clear();
        att_mt = 1;
    }
};

}  // namespace kvr

// Device scratch of kvr_select_attention_noalloc, a fixed file-scope array:
// each device the library runs on holds one copy until the process ends, and
// every call on that device shares it.  In host code `scratch` names a
// host-side stand-in, not the device copy: its device address comes from
// hipGetSymbolAddress, looked up once per device (scratch_address) and kept
// in each context; only that address is passed to kernels.
static constexpr size_t NOALLOC_SCRATCH_BYTES = 4u << 20;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

struct kvr_ctx {
    kvr_dims d{};
    int device = 0;
    bool bf16 = true;
    bool force_simple = false;
    std::vector<kvr_layer_weights> layers;
    const void *embed = nullptr, *final_norm = nullptr;

    // projection weights repacked in operand order (bf16 MFMA paths)
    struct PackedLayer { const void *qkv, *o, *gu, *down; };
    // tile group of each projection's packed weights (packed_tile_offset)
    int qkv_grp = 1, o_grp = 1, gu_grp = 1, down_grp = 1;
    std::vector<PackedLayer> pk;
    char *wpk = nullptr;
    size_t wpk_bytes = 0;

    // scoring: LM head (borrowed; the embedding when tied), its packed copy,
    // and buffers made on the first kvr_score / kvr_generate call
    const void *lm_head = nullptr;
    void *lm_pk = nullptr;
    size_t lm_pk_bytes = 0;
    char *sel_scratch = nullptr;  // selectors: CacheBlend fresh keys/values + deviations; Attention mass
    size_t sel_bytes = 0;
    float *score_y = nullptr;     // hidden rows of the scored block [max rows][d]
    float *score_part = nullptr;  // logit tiles [split][64][vocab]
    void *score_lsm = nullptr;    // log-softmax chunk statistics
    size_t score_bytes = 0;

    int rows_cap = 0;  // rows per pass
    int max_docs = 0;
    int items_cap = 0, comb_cap = 0;

    char *ws = nullptr;
    size_t ws_bytes = 0;
    float *H = nullptr, *P = nullptr;  // residual stream; projection outputs / split-K partials
    float *rs_ssq = nullptr;           // skinny passes: per-row sums of squares by column block (resid_gain)
    size_t p_floats = 0;               // capacity of P
    // matrix operands; in bf16 each is a compensated pair (hi, lo)
    void *Xn = nullptr, *Qb = nullptr, *Ob = nullptr, *Ab = nullptr;
    void *Xn_lo = nullptr, *Qb_lo = nullptr, *Ob_lo = nullptr, *Ab_lo = nullptr;
    float *rope_cos = nullptr, *rope_sin = nullptr;
    float *attn_part = nullptr;
    size_t attn_part_floats = 0;
    char *d_tables = nullptr;
    size_t tables_bytes = 0;
    Tables tab;  // host tables of the pass being planned (capacity reserved at create)
    void *scratch_ptr = nullptr;        // this device's copy of `scratch` (kvr_select_attention_noalloc)
    hipError_t scratch_err = hipSuccess;

    char *h_stage = nullptr;
    hipEvent_t stage_ev = nullptr;
    bool stage_pending = false;

    // per-step event profiling
    bool profiling = false;
    std::vector<hipEvent_t> ev_pool;
    struct Timed { int step; hipEvent_t start, stop; };
    std::vector<Timed> ev_marks;  // launches timed since the last read
    double step_ms[16] = {};
    long long step_n[16] = {};

    std::string err;
};

namespace {

constexpr int PREFILL_CHUNK = 8192;
constexpr size_t ATTN_PART_BYTES = 64ull << 20;
constexpr int PART_ROW = ATT_HD + 4;
constexpr int SPLIT_MAX = 32;

enum Step {
    ST_EMBED, ST_NORM, ST_QKV, ST_ROPE, ST_ATTN, ST_COMBINE, ST_OPROJ, ST_GATEUP, ST_DOWN, ST_FINAL, ST_LMHEAD,
    ST_LOGSOFTMAX, ST_MASS, ST_SWIGLU, ST_COUNT
};
const char *const STEP_NAMES[ST_COUNT] = {"embed", "rmsnorm", "qkv_proj", "rope_scatter", "attention",
                                          "attention_combine", "o_proj", "gate_up_swiglu", "down_proj", "final_norm",
                                          "lm_head", "logsoftmax", "attention_mass", "swiglu_partials"};
constexpr int SCORE_ROWS = 64;  // rows per LM-head launch (the skinny kernel's bound)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int env_int(const char *name, int dflt) {
    const char *v = name ? getenv(name) : nullptr;
    return (v && *v) ? atoi(v) : dflt;
}

kvr_status fail(kvr_ctx *c, kvr_status st, const std::string &msg) {
    if (c) c->err = msg;
    else kvr::set_global_error(msg.c_str());
    return st;
}

kvr_status hip_fail(kvr_ctx *c, hipError_t e, const char *what) {
    return fail(c, KVR_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Device address of `scratch` on the current device, looked up once per
// device (hipGetSymbolAddress with that device current) and kept.
hipError_t scratch_address(int device, void **out) {
    static std::mutex mu;
    static std::map<int, std::pair<void *, hipError_t>> table;
    std::lock_guard<std::mutex> lock(mu);
    auto it = table.find(device);
    if (it == table.end()) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        it = table.emplace(device, std::make_pair(e == hipSuccess ? ptr : nullptr, e)).first;
    }
    *out = it->second.first;
    return it->second.second;
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        int cur = 0;
        if (hipGetDevice(&cur) == hipSuccess && cur != dev && hipSetDevice(dev) == hipSuccess) prev = cur;
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

size_t elem_size(const kvr_dims &d) { return d.dtype == KVR_BF16 ? 2 : 4; }

// Split the key ranges of the row blocks over work items: without splitting
// when there are enough items to fill the GPU, otherwise in chunks of KS keys
// (a multiple of the 64-key tile, at least two tiles) so that about `target`
// items exist.  The attention kernel runs one block per compute unit, so the
// target is one item per unit: more, shorter items cost a second round and a
// longer combine (Mistral shape, 48 rows at 4900-4950: 0.92 ms of attention
// and combine per repair at 768 items against 0.64 ms at 256).
void plan_attention(const kvr_ctx *c, Tables &t) {
    const int Hkv = c->d.n_kv_heads;
    const int G = c->d.n_heads / Hkv;
    using Block = Tables::Block;
    std::vector<Block> &blocks = t.blocks;
    auto make_blocks = [&](int rows_blk) {
        blocks.clear();
        for (int di = 0; di < (int)t.docs.size(); ++di) {
            const DocInfo &dc = t.docs[di];
            for (int b = 0; b < dc.nrows; b += rows_blk) {
                const int nb = std::min(rows_blk, dc.nrows - b);
                blocks.push_back({di, dc.row0 + b, nb, t.rows[dc.row0 + b + nb - 1].pos + 1});
            }
        }
    };
    const int target_env = env_int("KVR_ATT_TARGET", 0);
    int target = target_env > 0 ? target_env : 256;
    const int mt_max = attention_max_row_tiles(c->d.n_heads, Hkv);
    int mt = mt_max;
    make_blocks(16 * mt);
    // Too few (row block, kv head) items to fill the GPU: split the key ranges.
    // The row blocks then shrink to one 16-row tile: the items of a key range
    // read the same K/V tiles (from L2), each row's keys are cut into fewer
    // parts (fewer partials to write and combine), and an item of one tile
    // has few enough (head, row tile) pairs for the kernel's two key groups.
    const bool split = (long long)blocks.size() * Hkv < target / 2;
    if (split) {
        mt = std::min(mt_max, std::max(1, env_int("KVR_ATT_MT", 1)));
        make_blocks(16 * mt);
    }
    t.att_mt = mt;
    const int rows_blk = 16 * mt;
    long long total_keys = 0;
    for (auto &b : blocks) total_keys += b.kmax;
    int KS = 1 << 30;
    const size_t slot_floats = (size_t)G * rows_blk * PART_ROW;
    const size_t max_slots = c->attn_part_floats / slot_floats;
    if (split) {
        long long ks = (total_keys * Hkv + target - 1) / target;
        // Items of a dozen key tiles or more (many rows: Qwen2.5-7B shape at
        // 528 rows, 17-tile items) run as twice as many half-length items:
        // the units that finish early take the rest, and the last round is
        // short (attention 59.5 -> 48.0 us per layer; at 144 rows, 5-tile
        // items, the doubled target cost 17.1 -> 23.0 us)
        if (target_env <= 0 && ks >= 12 * ATT_KT) {
            target *= 2;
            ks = (total_keys * Hkv + target - 1) / target;
        }
        ks = std::max<long long>(env_int("KVR_ATT_MINKS", 128), (ks + ATT_KT - 1) / ATT_KT * ATT_KT);
        for (;; ks *= 2) {
            size_t slots = 0, nitems = 0;
            for (auto &b : blocks) {
                const long long ns = (b.kmax + ks - 1) / ks;
                nitems += (size_t)ns * Hkv;
                if (ns > 1) slots += (size_t)ns * Hkv;
            }
            if (slots <= max_slots && nitems <= (size_t)c->items_cap) break;
        }
        KS = (int)std::min<long long>(ks, 1 << 30);
    }
    int next_slot = 0;
    for (auto &b : blocks) {
        const int ns = (b.kmax + KS - 1) / KS;
        for (int g = 0; g < Hkv; ++g) {
            if (ns <= 1) {
                t.items.push_back({b.doc, b.row0, b.nrows, g, 0, b.kmax, -1, t.docs[b.doc].n_cap, t.docs[b.doc].cache});
                continue;
            }
            CombineItem ci{};
            ci.row0 = b.row0; ci.nrows = b.nrows; ci.kvh = g; ci.part0 = next_slot; ci.nparts = ns;
            t.comb.push_back(ci);
            for (int s = 0; s < ns; ++s)
                t.items.push_back({b.doc, b.row0, b.nrows, g, s * KS, std::min(b.kmax, (s + 1) * KS), next_slot + s,
                                   t.docs[b.doc].n_cap, t.docs[b.doc].cache});
            next_slot += ns;
        }
    }
    // longest key ranges first, so that short items fill the tail; equal
    // lengths keep the order they were made in (document, rows, kv head, keys),
    // which is a total order, so the in-place sort is deterministic
    std::sort(t.items.begin(), t.items.end(), [](const AttnItem &x, const AttnItem &y) {
        if (x.k1 - x.k0 != y.k1 - y.k0) return (x.k1 - x.k0) > (y.k1 - y.k0);
        if (x.row0 != y.row0) return x.row0 < y.row0;
        if (x.kvh != y.kvh) return x.kvh < y.kvh;
        return x.k0 < y.k0;
    });
}

// Weight tiles per block and split-K factor of a skinny projection.  The X
// operand is re-read from L2 once per block column, so blocks are wide; a
// block streams NT tiles over its K slice, and blocks beyond one per compute
// unit run in a further round.  The plan minimises
//   rounds * NT * k-steps per slice,   rounds = ceil(blocks / 256),
// over NT <= 10 (7 for 64 rows, whose accumulators would spill at 8 and
// whose wavefronts' partial sums would not fit in LDS beyond 8) and
// splits up to the largest power of two that keeps each wavefront's K slice
// above `wave_ks` k-steps (and at least 7, which lets the Qwen2.5-7B output
// projection's 112 k-steps take 4 x 4: 0.312 -> 0.293 ms per repair), never
// splitting SwiGLU; ties go to
// the wider block, then the smaller split.  wave_ks is 16 for the QKV
// projection and the LM head and 8 for the output and down projections.
// Measured on the 8B shape this reproduces the best of the swept plans
// (QKV 3 x 2, O 4 x 4, gate/up 7, down 8 x 8); on the Qwen2.5-7B shape it
// takes gate/up 10 (237 blocks in one round, tied with 5 in two rounds of
// 474: each block reads the whole activation matrix from L2, so the wider
// block halves that traffic; 48 rows: 1.70 -> 1.45 ms per repair, against
// 2.12 ms at 8, 296 blocks) and down 7 x 8 (32 us against 43 us at 8 x 16).
struct SkinnyPlan { int nt, split; };

SkinnyPlan plan_skinny(int ntiles, int K, int R, bool swiglu, int wave_ks, const char *env_nt,
                       const char *env_split) {
    const int ksteps = K / 32;
    int smax = 1;
    if (!swiglu)
        while (smax * 2 <= SPLIT_MAX && ksteps / (4 * smax) > wave_ks && ksteps / (8 * smax) >= 7) smax *= 2;
    const int ntmax = (R + 15) / 16 >= 4 ? 7 : 10;
    SkinnyPlan p{1, 1};
    long long best = -1;
    for (int sp = 1; sp <= smax; sp *= 2)
        for (int nt = 1; nt <= ntmax; ++nt) {
            const long long blocks = (long long)((ntiles + nt - 1) / nt) * sp;
            const long long cost = (blocks + 255) / 256 * nt * ((ksteps + sp - 1) / sp);
            if (best < 0 || cost < best || (cost == best && nt > p.nt)) {
                p = SkinnyPlan{nt, sp};
                best = cost;
            }
        }
    const int es = env_split ? env_int(env_split, 0) : 0;
    if (!swiglu && es >= 1) p.split = std::min(es, std::min(SPLIT_MAX, ksteps));
    const int nt = env_int(env_nt, 0);
    if (nt >= 1 && nt <= ((R + 15) / 16 <= 3 ? 10 : 8)) p.nt = nt;
    return p;
}

// Shapes the packed-weight MFMA kernels take (K of every projection a multiple
// of 64, weight tiles of 16 rows).
bool pack_ok(const kvr_dims &d, bool force_simple) {
    const int qd = d.n_heads * d.head_dim, kd = d.n_kv_heads * d.head_dim;
    return d.dtype == KVR_BF16 && !force_simple && d.d_model % 64 == 0 && qd % 64 == 0 && d.d_ffn % 64 == 0 &&
           kd % 16 == 0;
}

bool skinny_pass_ok(const kvr_ctx *c, int R) { return c->wpk != nullptr && R <= 64; }

// Packed weight: the tiled MFMA kernel, whose activations are in operand
// order; otherwise the row-major simple kernel.
hipError_t linear(kvr_ctx *c, int epi, LinearArgs a, hipStream_t s) {
    if (a.wp && a.tpb > 0) return launch_linear_tall(epi, a, s);
    if (a.wp) return launch_linear_tiled(epi, a, s);
    return launch_linear_simple(c->bf16, epi, a, s);
}

LinearArgs make_args(const void *x, const void *x_lo, int ldx, int R, int K, int N, const void *w0, const void *w1,
                     const void *w2, int e0, int e1, const void *wp, void *out, void *out_lo, int ldo) {
    LinearArgs a{};
    a.x = x; a.x_lo = x_lo; a.ldx = ldx; a.R = R; a.K = K; a.N = N;
    a.out_lo = out_lo;
    a.w[0] = w0; a.w[1] = w1; a.w[2] = w2;
    a.seg_end[0] = e0; a.seg_end[1] = e1; a.seg_end[2] = N;
    a.wp = wp;
    a.grp = 1;
    a.out = out; a.ldo = ldo;
    a.split = 1;
    return a;
}

// rs_ssq: the rows' sums of squares from resid_gain (X is H * gain, not yet
// normalised): the kernel applies the RMS scale to its output rows.
hipError_t skinny(int epi, const void *x, const void *x_lo, int R, int K, int N, const void *wp, int grp, void *out,
                  void *out_lo, const SkinnyPlan &p, hipStream_t s, const float *rs_ssq = nullptr,
                  float rs_eps = 0.f) {
    SkinnyArgs a{};
    a.x = x; a.x_lo = x_lo; a.R = R; a.K = K; a.N = N;
    a.w = wp;
    a.grp = grp;
    a.rs_ssq = rs_ssq;
    a.rs_nb = resid_gain_blocks(K);
    a.rs_d = K;
    a.rs_eps = rs_eps;
    a.ntiles = (epi == EPI_SWIGLU ? 2 * N : N) / 16;
    a.out = out; a.out_lo = out_lo; a.split = p.split;
    return launch_linear_skinny(epi, a, p.nt, s);
}

// K slices for a tiled projection of R rows into vrows outputs whose partial
// tiles go to P: enough blocks for about two per compute unit, at least 16
// k-steps per slice, and no more partial tiles than P holds (1: no split).
int tiled_split(const kvr_ctx *c, int R, int vrows, int K) {
    int slots = 0;
    const int blocks = tiled_blocks(R, vrows, &slots);
    if (blocks >= 2 * 256) return 1;
    int split = (2 * 256 + blocks - 1) / blocks;
    split = std::min(split, std::max(1, K / 32 / 16));
    split = std::min<long long>(split, (long long)(c->p_floats / ((size_t)R * vrows)));
    return std::max(1, std::min(split, SPLIT_MAX));
}

// Kernel and K split of a packed-weight projection outside skinny passes: the
// tall kernel for 64 < R <= 192 rows, the tiled kernel otherwise (split for
// STORE projections only).  A tall SwiGLU plan with split > 1 runs as a STORE
// launch into P followed by the SwiGLU pass (run_pass).  Environment
// overrides of the tall plan: KVR_TALL=0 (tiled kernel instead),
// KVR_TALL_TPB (tiles per block), KVR_TALL_SPLIT (STORE split),
// KVR_TALL_GU_SPLIT (SwiGLU split, 1 or 2), KVR_TALL_STORE_TPB (widest STORE
// block the planner may take, 12-20).
void plan_packed(const kvr_ctx *c, LinearArgs &a, int epi) {
    const int vrows = epi == EPI_SWIGLU ? 2 * a.N : a.N;
    a.tpb = 0;
    a.split = 1;
    if (!a.wp) return;
    if (tall_rows_ok(a.R) && env_int("KVR_TALL", 1) != 0) {
        const bool gu = epi == EPI_SWIGLU;
        const int store_max = std::min(TALL_TPB_WIDE, std::max(TALL_TPB, env_int("KVR_TALL_STORE_TPB", TALL_TPB)));
        TallPlan p = plan_tall(a.R, vrows, a.K, gu, c->p_floats, store_max);
        const int gsp = gu ? env_int("KVR_TALL_GU_SPLIT", 0) : 0;
        if (gsp >= 1 && gsp <= TALL_GU_SPLIT_MAX && (size_t)gsp * a.R * vrows <= c->p_floats) {
            p.split = gsp;
            p.tpb = std::max(1, std::min(gsp == 1 ? TALL_TPB : TALL_TPB_WIDE, (vrows / 16 * gsp + 255) / 256));
        }
        const int tpb = env_int("KVR_TALL_TPB", 0), sp = env_int("KVR_TALL_SPLIT", 0);
        if (tpb >= 1 && tpb <= ((gu && p.split == 1) ? TALL_TPB : TALL_TPB_WIDE)) p.tpb = tpb;
        if (sp >= 1 && !gu && (size_t)sp * a.R * vrows <= c->p_floats)
            p.split = std::min(sp, std::min(TALL_SPLIT_MAX, a.K / 32));
        a.tpb = p.tpb;
        a.split = p.split;
        return;
    }
    if (epi == EPI_STORE) a.split = tiled_split(c, a.R, vrows, a.K);
}

// A tall projection reading the RMSNorm output applies the RMS scale to its
// output rows, as the skinny kernels do: the residual step then runs over
// (row, column block) blocks (resid_gain) instead of one block per row, whose
// 144 blocks at 144 rows leave compute units idle while they sum the output
// projection's partial tiles.  KVR_TALL_ROWSCALE=0 keeps the per-row kernel.
bool tall_row_scale(const LinearArgs &a) { return a.tpb > 0 && a.x_lo && env_int("KVR_TALL_ROWSCALE", 1) != 0; }

void set_row_scale(LinearArgs &a, const float *ssq, int K, float eps) {
    a.rs_ssq = ssq;
    a.rs_nb = resid_gain_blocks(K);
    a.rs_d = K;
    a.rs_eps = eps;
}

// Step profiler: arm() hands two events to the next kernel launch, which
// records them around its execution; disarm() files them under `step` (or
// returns them when the launcher enqueued nothing).
hipError_t take_event(kvr_ctx *c, hipEvent_t *ev) {
    if (!c->ev_pool.empty()) {
        *ev = c->ev_pool.back();
        c->ev_pool.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(ev);
}

hipError_t arm(kvr_ctx *c) {
    if (!c->profiling) return hipSuccess;
    LaunchTimer &t = launch_timer();
    hipError_t e = take_event(c, &t.start);
    if (e == hipSuccess) e = take_event(c, &t.stop);
    return e;
}

void disarm(kvr_ctx *c, int step, hipEvent_t start, hipEvent_t stop) {
    if (!c->profiling || !start) return;
    LaunchTimer &t = launch_timer();
    if (t.start == nullptr) {
        c->ev_marks.push_back({step, start, stop});  // consumed by a launch
    } else {
        c->ev_pool.push_back(start);
        c->ev_pool.push_back(stop);
        t.start = t.stop = nullptr;
    }
}

// Attention-mass accumulation during a pass of query rows (Attention
// selector): after each layer's attention the probability mass the pass's
// rows place on the stale keys [0, n) is added to part [Hkv][n]; the pass ends
// after the last layer's attention.
struct MassHook {
    const void *cache;
    int n_cap, n;
    float *lse;   // [rows][Hq]
    float *part;  // [Hkv][n]
};

// Upload the tables of a pass and enqueue its kernels.  kv_layer >= 0 stops
// the pass at that layer once its fresh keys/values are in the cache (layers
// below it run in full; no final norm).
kvr_status run_pass(kvr_ctx *c, Tables &t, hipStream_t s, int kv_layer = -1, const MassHook *mh = nullptr) {
    const kvr_dims &d = c->d;
    const int R = (int)t.rows.size();
    if (R == 0) return KVR_OK;
    const bool attn_mfma = c->bf16 && !c->force_simple && d.head_dim == ATT_HD && d.n_heads / d.n_kv_heads <= 16;
    const bool sk = skinny_pass_ok(c, R);
    const bool op = c->wpk != nullptr;  // matrix operands in MFMA operand order (both packed-weight kernels)
    if (attn_mfma) plan_attention(c, t);
    if ((int)t.items.size() > c->items_cap || (int)t.comb.size() > c->comb_cap)
        return fail(c, KVR_E_RANGE, "attention plan exceeds the context's item capacity");

    // pack the tables: rows | docs | items | combine
    const size_t o_docs = align_up(t.rows.size() * sizeof(RowInfo), 256);
    const size_t o_items = o_docs + align_up(t.docs.size() * sizeof(DocInfo), 256);
    const size_t o_comb = o_items + align_up(t.items.size() * sizeof(AttnItem), 256);
    const size_t total = o_comb + t.comb.size() * sizeof(CombineItem);
    if (total > c->tables_bytes) return fail(c, KVR_E_RANGE, "pass tables exceed the context's staging capacity");
    if (c->stage_pending) {
        hipError_t e = hipEventSynchronize(c->stage_ev);
        if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize(staging)");
        c->stage_pending = false;
    }
    memcpy(c->h_stage, t.rows.data(), t.rows.size() * sizeof(RowInfo));
    memcpy(c->h_stage + o_docs, t.docs.data(), t.docs.size() * sizeof(DocInfo));
    if (!t.items.empty()) memcpy(c->h_stage + o_items, t.items.data(), t.items.size() * sizeof(AttnItem));
    if (!t.comb.empty()) memcpy(c->h_stage + o_comb, t.comb.data(), t.comb.size() * sizeof(CombineItem));
    hipError_t e = hipMemcpyAsync(c->d_tables, c->h_stage, total, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(c, e, "hipMemcpyAsync(tables)");
    e = hipEventRecord(c->stage_ev, s);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventRecord(staging)");
    c->stage_pending = true;
    const RowInfo *rows = (const RowInfo *)c->d_tables;
    const DocInfo *docs = (const DocInfo *)(c->d_tables + o_docs);
    const AttnItem *items = (const AttnItem *)(c->d_tables + o_items);
    const CombineItem *comb = (const CombineItem *)(c->d_tables + o_comb);

    const int D = d.d_model, F = d.d_ffn, hd = d.head_dim;
    const int qd = d.n_heads * hd, kd = d.n_kv_heads * hd, NQKV = qd + 2 * kd;
    const bool bf = c->bf16;
    SkinnyPlan p_qkv{}, p_o{}, p_gu{}, p_down{};
    if (sk) {
        // QKV at 6 tiles x split 4 ran 0.3 us faster than 3 x 2 but doubled the
        // partials RoPE/scatter sums (0.4 us slower): the K slices stay long
        p_qkv = plan_skinny(NQKV / 16, D, R, false, 16, "KVR_NT_QKV", "KVR_SPLIT_QKV");
        p_o = plan_skinny(D / 16, qd, R, false, 8, "KVR_NT_O", "KVR_SPLIT_O");
        p_gu = plan_skinny(2 * F / 16, D, R, true, 16, "KVR_NT_GATEUP", nullptr);
        p_down = plan_skinny(D / 16, F, R, false, 8, "KVR_NT_DOWN", "KVR_SPLIT_DOWN");
    }
#define KVR_CHECK(expr, what, step)                                                \
    do {                                                                           \
        hipError_t err_ = arm(c);                                                  \
        const LaunchTimer armed_ = launch_timer();                                 \
        if (err_ == hipSuccess) err_ = (expr);                                     \
        disarm(c, step, armed_.start, armed_.stop);                                \
        if (err_ != hipSuccess) return hip_fail(c, err_, what);                    \
    } while (0)

    KVR_CHECK(launch_embed(bf, rows, docs, R, c->embed, D, d.vocab, c->H, s), "embed", ST_EMBED);
    int resid_split = 0;  // partial tiles in P still to be added to H
    const int n_run = kv_layer >= 0 ? kv_layer + 1 : d.n_layers;
    for (int l = 0; l < n_run; ++l) {
        const kvr_layer_weights &w = c->layers[l];
        const kvr_ctx::PackedLayer pw = c->wpk ? c->pk[l] : kvr_ctx::PackedLayer{nullptr, nullptr, nullptr, nullptr};
        // skinny and tall passes: the projections apply the RMS scale to their
        // outputs (resid_gain spreads the residual step over column blocks)
        LinearArgs qa{};
        bool rg = sk;
        if (!sk) {
            qa = make_args(c->Xn, c->Xn_lo, D, R, D, NQKV, w.wq, w.wk, w.wv, qd, qd + kd, pw.qkv, c->P, nullptr, NQKV);
            qa.grp = c->qkv_grp;
            plan_packed(c, qa, EPI_STORE);
            rg = tall_row_scale(qa);
        }
        if (rg)
            KVR_CHECK(launch_resid_gain(bf, c->H, c->P, resid_split, w.attn_norm, R, D, c->Xn, c->Xn_lo, c->rs_ssq, s),
                      "rmsnorm(attn)", ST_NORM);
        else
            KVR_CHECK(launch_rmsnorm(bf, bf, c->H, c->P, resid_split, w.attn_norm, R, D, d.rms_eps, c->Xn, c->Xn_lo, D,
                                     op, s),
                      "rmsnorm(attn)", ST_NORM);
        int qkv_split = 1;
        if (sk) {
            KVR_CHECK(skinny(EPI_STORE, c->Xn, c->Xn_lo, R, D, NQKV, pw.qkv, c->qkv_grp, c->P, nullptr, p_qkv, s, c->rs_ssq,
                             d.rms_eps),
                      "qkv", ST_QKV);
            qkv_split = p_qkv.split;
        } else {
            if (rg) set_row_scale(qa, c->rs_ssq, D, d.rms_eps);
            KVR_CHECK(linear(c, EPI_STORE, qa, s), "qkv", ST_QKV);
            qkv_split = qa.split;
        }
        KVR_CHECK(launch_rope_scatter(bf, c->P, qkv_split, w.bq, w.bk, w.bv, rows, docs, R, l, d.n_heads, d.n_kv_heads,
                                      hd, c->rope_cos, c->rope_sin, c->Qb, c->Qb_lo, s), "rope_scatter", ST_ROPE);
        if (l == kv_layer) return KVR_OK;
        float *lse = mh ? mh->lse : nullptr;
        if (attn_mfma) {
            KVR_CHECK(launch_attention_mfma((const bf16_t *)c->Qb, (const bf16_t *)c->Qb_lo, rows, items,
                                            (int)t.items.size(), t.att_mt, l, d.n_heads, d.n_kv_heads, c->attn_part,
                                            (bf16_t *)c->Ob, (bf16_t *)c->Ob_lo, op, lse, s),
                      "attention", ST_ATTN);
            if (!t.comb.empty())
                KVR_CHECK(launch_attention_combine(comb, (int)t.comb.size(), t.att_mt, c->attn_part, d.n_heads, d.n_kv_heads,
                                                   (bf16_t *)c->Ob, (bf16_t *)c->Ob_lo, op, lse, s), "attention_combine", ST_COMBINE);
        } else {
            KVR_CHECK(launch_attention_simple(bf, c->Qb, c->Qb_lo, rows, docs, R, l, d.n_heads, d.n_kv_heads, hd, c->Ob,
                                              c->Ob_lo, op, lse, s),
                      "attention_simple", ST_ATTN);
        }
        if (mh) {
            KVR_CHECK(launch_attn_mass(bf, c->Qb, c->Qb_lo, mh->lse, R, mh->cache, mh->n_cap, l, d.n_heads,
                                       d.n_kv_heads, hd, mh->n, mh->part, l > 0, s),
                      "attention_mass", ST_MASS);
            if (l == d.n_layers - 1) return KVR_OK;
        }
        if (sk) {
            KVR_CHECK(skinny(EPI_STORE, c->Ob, c->Ob_lo, R, qd, D, pw.o, c->o_grp, c->P, nullptr, p_o, s), "o_proj", ST_OPROJ);
            resid_split = p_o.split;
        } else if (pw.o) {
            // packed: partial tiles into P (the next RMSNorm adds them to H)
            LinearArgs a = make_args(c->Ob, c->Ob_lo, qd, R, qd, D, w.wo, w.wo, w.wo, D, D, pw.o, c->P, nullptr, D);
            a.grp = c->o_grp;
            plan_packed(c, a, EPI_STORE);
            KVR_CHECK(linear(c, EPI_STORE, a, s), "o_proj", ST_OPROJ);
            resid_split = a.split;
        } else {
            KVR_CHECK(linear(c, EPI_RESID, make_args(c->Ob, c->Ob_lo, qd, R, qd, D, w.wo, w.wo, w.wo, D, D, pw.o, c->H, nullptr, D), s),
                      "o_proj", ST_OPROJ);
        }
        LinearArgs ga{};
        rg = sk;
        if (!sk) {
            ga = make_args(c->Xn, c->Xn_lo, D, R, D, F, w.w_gate, w.w_up, w.w_up, F, F, pw.gu, c->Ab, c->Ab_lo, F);
            ga.grp = c->gu_grp;
            plan_packed(c, ga, EPI_SWIGLU);
            rg = tall_row_scale(ga);
        }
        if (rg)
            KVR_CHECK(launch_resid_gain(bf, c->H, c->P, resid_split, w.mlp_norm, R, D, c->Xn, c->Xn_lo, c->rs_ssq, s),
                      "rmsnorm(mlp)", ST_NORM);
        else
            KVR_CHECK(launch_rmsnorm(bf, bf, c->H, c->P, resid_split, w.mlp_norm, R, D, d.rms_eps, c->Xn, c->Xn_lo, D, op,
                                     s),
                      "rmsnorm(mlp)", ST_NORM);
        resid_split = 0;
        if (sk) {
            KVR_CHECK(skinny(EPI_SWIGLU, c->Xn, c->Xn_lo, R, D, F, pw.gu, c->gu_grp, c->Ab, c->Ab_lo, p_gu, s, c->rs_ssq,
                             d.rms_eps),
                      "gate_up", ST_GATEUP);
            KVR_CHECK(skinny(EPI_STORE, c->Ab, c->Ab_lo, R, F, D, pw.down, c->down_grp, c->P, nullptr, p_down, s), "down",
                      ST_DOWN);
            resid_split = p_down.split;
        } else {
            if (rg) set_row_scale(ga, c->rs_ssq, D, d.rms_eps);
            if (ga.tpb > 0 && ga.split > 1) {
                // split gate/up (tall): fp32 partials of the 2F interleaved
                // columns into P (free: the residual step consumed the output
                // projection's), then the SwiGLU pass writes the down
                // projection's operand
                LinearArgs pa = ga;
                pa.N = 2 * F;
                pa.out = c->P;
                pa.out_lo = nullptr;
                pa.ldo = 2 * F;
                KVR_CHECK(launch_linear_tall(EPI_STORE, pa, s), "gate_up", ST_GATEUP);
                KVR_CHECK(launch_swiglu_partials(c->P, ga.split, R, F, (bf16_t *)c->Ab, (bf16_t *)c->Ab_lo, s),
                          "swiglu_partials", ST_SWIGLU);
            } else {
                KVR_CHECK(linear(c, EPI_SWIGLU, ga, s), "gate_up", ST_GATEUP);
            }
            if (pw.down) {
                LinearArgs a = make_args(c->Ab, c->Ab_lo, F, R, F, D, w.w_down, w.w_down, w.w_down, D, D, pw.down, c->P,
                                         nullptr, D);
                a.grp = c->down_grp;
                plan_packed(c, a, EPI_STORE);
                KVR_CHECK(linear(c, EPI_STORE, a, s), "down", ST_DOWN);
                resid_split = a.split;
            } else {
                KVR_CHECK(linear(c, EPI_RESID, make_args(c->Ab, c->Ab_lo, F, R, F, D, w.w_down, w.w_down, w.w_down, D, D,
                                                         pw.down, c->H, nullptr, D), s),
                          "down", ST_DOWN);
            }
        }
    }
    KVR_CHECK(launch_final_norm(bf, c->H, c->P, resid_split, c->final_norm, rows, docs, R, D, d.rms_eps, s),
              "final_norm", ST_FINAL);
#undef KVR_CHECK
    return KVR_OK;
}

// Forward over the m rows at positions [n, n+m) of one document (their keys
// and values land in cache slots [n, n+m)), then the LM head and the
// log-softmax in blocks of SCORE_ROWS rows: lp[j] = log p(tokens[n+j+1]) for
// j < m-1, argmax[j] for j < m, and *next = argmax of row m-1.
kvr_status score_block(kvr_ctx *c, void *cache, int n, int n_cap, const int32_t *tokens, int m, float *lp,
                       int32_t *argmax, int32_t *next, hipStream_t s) {
    const kvr_dims &d = c->d;
    const int D = d.d_model, V = d.vocab;
    Tables &t = c->tab;
    t.clear();
    t.docs.push_back(DocInfo{cache, tokens, c->score_y, n + m, n_cap, 0, m});
    t.rows.reserve(m);
    for (int j = 0; j < m; ++j) t.rows.push_back(RowInfo{n + j, 0, j, 0});
    kvr_status st = run_pass(c, t, s);
    if (st != KVR_OK) return st;
    const SkinnyPlan plan = plan_skinny(V / 16, D, SCORE_ROWS, false, 16, "KVR_NT_LM", "KVR_SPLIT_LM");
#define KVR_SCHECK(expr, what, step)                                                \
    do {                                                                           \
        hipError_t err_ = arm(c);                                                  \
        const LaunchTimer armed_ = launch_timer();                                 \
        if (err_ == hipSuccess) err_ = (expr);                                     \
        disarm(c, step, armed_.start, armed_.stop);                                \
        if (err_ != hipSuccess) return hip_fail(c, err_, what);                    \
    } while (0)
    for (int c0 = 0; c0 < m; c0 += SCORE_ROWS) {
        const int R = std::min(SCORE_ROWS, m - c0);
        const float *Y = c->score_y + (size_t)c0 * D;
        int nsplit = 1;
        if (c->lm_pk) {
            KVR_SCHECK(launch_to_operand(true, true, Y, R, D, c->Xn, c->Xn_lo, s), "lm_head operand", ST_LMHEAD);
            KVR_SCHECK(skinny(EPI_STORE, c->Xn, c->Xn_lo, R, D, V, c->lm_pk, 1, c->score_part, nullptr, plan, s),
                       "lm_head", ST_LMHEAD);
            nsplit = plan.split;
        } else if (c->bf16) {
            KVR_SCHECK(launch_to_operand(true, false, Y, R, D, c->Xn, c->Xn_lo, s), "lm_head operand", ST_LMHEAD);
            KVR_SCHECK(launch_linear_simple(true, EPI_STORE, make_args(c->Xn, c->Xn_lo, D, R, D, V, c->lm_head,
                                                                       c->lm_head, c->lm_head, V, V, nullptr,
                                                                       c->score_part, nullptr, V), s),
                       "lm_head", ST_LMHEAD);
        } else {
            KVR_SCHECK(launch_linear_simple(false, EPI_STORE, make_args(Y, nullptr, D, R, D, V, c->lm_head, c->lm_head,
                                                                        c->lm_head, V, V, nullptr, c->score_part,
                                                                        nullptr, V), s),
                       "lm_head", ST_LMHEAD);
        }
        const int nt = lp ? std::max(0, std::min(R, m - 1 - c0)) : 0;  // rows with a target to score
        KVR_SCHECK(launch_logsoftmax(c->score_part, nsplit, R, V, tokens + n + c0 + 1, nt, lp ? lp + c0 : nullptr,
                                     argmax ? argmax + c0 : nullptr, (c0 + R == m) ? next : nullptr, c->score_lsm, s),
                   "logsoftmax", ST_LOGSOFTMAX);
    }
#undef KVR_SCHECK
    return KVR_OK;
}

kvr_status score_buffers(kvr_ctx *c) {
    if (c->score_y) return KVR_OK;
    const kvr_dims &d = c->d;
    const SkinnyPlan plan = plan_skinny(d.vocab / 16, d.d_model, SCORE_ROWS, false, 16, "KVR_NT_LM", "KVR_SPLIT_LM");
    const size_t y_bytes = align_up((size_t)c->rows_cap * d.d_model * 4, 256);
    const size_t p_bytes = align_up((size_t)std::max(plan.split, 1) * SCORE_ROWS * d.vocab * 4, 256);
    const size_t l_bytes = logsoftmax_ws_bytes(SCORE_ROWS, d.vocab);
    char *buf = nullptr;
    hipError_t e = hipMalloc((void **)&buf, y_bytes + p_bytes + l_bytes);
    if (e != hipSuccess) return fail(c, KVR_E_NOMEM, "scoring buffer allocation failed");
    c->score_y = (float *)buf;
    c->score_part = (float *)(buf + y_bytes);
    c->score_lsm = buf + y_bytes + p_bytes;
    c->score_bytes = y_bytes + p_bytes + l_bytes;
    return KVR_OK;
}

kvr_status check_dims(const kvr_dims *d) {
    if (!d) return KVR_E_ARG;
    if (d->n_layers < 1 || d->d_model < 1 || d->n_heads < 1 || d->n_kv_heads < 1 || d->head_dim < 2 ||
        d->d_ffn < 1 || d->vocab < 1 || d->max_ctx < 1 || d->max_rows < 1)
        return KVR_E_ARG;
    if (d->n_heads % d->n_kv_heads != 0 || d->head_dim % 2 != 0) return KVR_E_ARG;
    if (!(d->rms_eps >= 0.f) || !(d->rope_theta > 0.0)) return KVR_E_ARG;
    if (d->dtype != KVR_F32 && d->dtype != KVR_BF16) return KVR_E_ARG;
    if (d->head_dim > 128) return KVR_E_UNSUPPORTED;
    // the row kernels move four floats per access over d_model (at most 16384)
    // and over the fused Q|K|V row of (n_heads + 2 n_kv_heads) head_dim values
    if (d->d_model % 4 != 0 || d->d_model > 16384 || ((d->n_heads + 2 * d->n_kv_heads) * d->head_dim) % 4 != 0)
        return KVR_E_UNSUPPORTED;
    return KVR_OK;
}

}  // namespace

extern "C" {

size_t kvr_cache_bytes(const kvr_dims *d, int32_t n_cap) {
    if (!d || n_cap < 0 || check_dims(d) != KVR_OK) return 0;
    return (size_t)d->n_layers * 2 * d->n_kv_heads * (size_t)n_cap * d->head_dim * elem_size(*d);
}

size_t kvr_workspace_bytes(const kvr_ctx *c) {
    return c ? c->ws_bytes + c->wpk_bytes + c->lm_pk_bytes + c->score_bytes + c->sel_bytes : 0;
}

const char *kvr_last_error(const kvr_ctx *c) { return c ? c->err.c_str() : g_error.c_str(); }

kvr_status kvr_create(const kvr_dims *dims, const kvr_weights *wts, kvr_ctx **out) {
    if (!out) return fail(nullptr, KVR_E_ARG, "kvr_create: out is NULL");
    *out = nullptr;
    kvr_status st = check_dims(dims);
    if (st != KVR_OK)
        return fail(nullptr, st, st == KVR_E_UNSUPPORTED ? "kvr_create: head_dim > 128 is not supported"
                                                         : "kvr_create: invalid dims");
    if (!wts || !wts->embed || !wts->final_norm || !wts->layers)
        return fail(nullptr, KVR_E_ARG, "kvr_create: NULL weights");
    const kvr_dims &d = *dims;
    if (!aligned16(wts->embed) || !aligned16(wts->final_norm) || (wts->lm_head && !aligned16(wts->lm_head)))
        return fail(nullptr, KVR_E_ARG, "kvr_create: weights must be 16-byte aligned");
    for (int l = 0; l < d.n_layers; ++l) {
        const kvr_layer_weights &w = wts->layers[l];
        const void *req[] = {w.attn_norm, w.wq, w.wk, w.wv, w.wo, w.mlp_norm, w.w_gate, w.w_up, w.w_down};
        for (const void *p : req)
            if (!p || !aligned16(p)) return fail(nullptr, KVR_E_ARG, "kvr_create: missing or misaligned layer weight");
        const void *bias[] = {w.bq, w.bk, w.bv};
        for (const void *p : bias) {
            if (d.qkv_bias && (!p || !aligned16(p)))
                return fail(nullptr, KVR_E_ARG, "kvr_create: qkv_bias set but a bias is missing or misaligned");
            if (!d.qkv_bias && p) return fail(nullptr, KVR_E_ARG, "kvr_create: bias given but qkv_bias is 0");
        }
    }

    kvr_ctx *c = new kvr_ctx();
    c->d = d;
    c->bf16 = d.dtype == KVR_BF16;
    const char *fs = getenv("KVR_SIMPLE");
    c->force_simple = fs && fs[0] == '1';
    c->layers.assign(wts->layers, wts->layers + d.n_layers);
    c->embed = wts->embed;
    c->final_norm = wts->final_norm;
    c->lm_head = wts->lm_head ? wts->lm_head : wts->embed;
    hipError_t e = hipGetDevice(&c->device);
    if (e != hipSuccess) { delete c; return hip_fail(nullptr, e, "hipGetDevice"); }
    // the no-allocation selector's scratch on this (current) device; a failed
    // lookup only disables that entry point
    c->scratch_err = scratch_address(c->device, &c->scratch_ptr);

    const int D = d.d_model, F = d.d_ffn, hd = d.head_dim;
    const int qd = d.n_heads * hd, kd = d.n_kv_heads * hd;
    const size_t es = elem_size(d);
    c->rows_cap = std::max(d.max_rows, std::min(d.max_ctx, PREFILL_CHUNK));
    c->max_docs = std::max(1, d.max_rows);
    const int G = d.n_heads / d.n_kv_heads;
    c->attn_part_floats = ATTN_PART_BYTES / 4;
    const size_t slot_floats = (size_t)G * 16 * PART_ROW;
    const int max_slots = (int)(c->attn_part_floats / slot_floats);
    const int blocks_cap = c->rows_cap / 16 + c->max_docs + 1;
    c->items_cap = blocks_cap * d.n_kv_heads + max_slots;
    c->comb_cap = blocks_cap * d.n_kv_heads;
    c->tab.rows.reserve(c->rows_cap);
    c->tab.docs.reserve(c->max_docs);
    c->tab.items.reserve(c->items_cap);
    c->tab.comb.reserve(c->comb_cap);
    c->tab.blocks.reserve(blocks_cap);
    c->tables_bytes = align_up((size_t)c->rows_cap * sizeof(RowInfo), 256) +
                      align_up((size_t)c->max_docs * sizeof(DocInfo), 256) +
                      align_up((size_t)c->items_cap * sizeof(AttnItem), 256) + (size_t)c->comb_cap * sizeof(CombineItem);

    const size_t R = align_up((size_t)c->rows_cap, 64);
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
    // P also takes a split tall gate/up projection's partials (passes of 65-192 rows)
    const size_t tall_rows = c->rows_cap > 64 ? std::min<size_t>(R, 16 * TALL_MT_MAX) : 0;
    const size_t p_floats = std::max({R * (qd + 2 * kd), (size_t)SPLIT_MAX * 64 * std::max(qd + 2 * kd, D),
                                      (size_t)TALL_GU_SPLIT_MAX * tall_rows * 2 * F});
    const size_t lo_es = c->bf16 ? es : 0;  // compensated low parts exist in bf16 only
    const size_t o_H = take(R * D * 4), o_P = take(p_floats * 4), o_Xn = take(R * D * es),
                 o_Qb = take(R * qd * es), o_Ob = take(R * qd * es), o_Ab = take(R * F * es),
                 o_Xl = take(R * D * lo_es), o_Ql = take(R * qd * lo_es), o_Ol = take(R * qd * lo_es),
                 o_Al = take(R * F * lo_es),
                 o_cos = take((size_t)d.max_ctx * (hd / 2) * 4), o_sin = take((size_t)d.max_ctx * (hd / 2) * 4),
                 o_ap = take(c->attn_part_floats * 4), o_tab = take(c->tables_bytes),
                 o_ss = take(std::max<size_t>(64, tall_rows) * resid_gain_blocks(D) * 4);
    c->ws_bytes = off;
    e = hipMalloc((void **)&c->ws, c->ws_bytes);
    if (e != hipSuccess) { delete c; return fail(nullptr, KVR_E_NOMEM, "kvr_create: workspace allocation failed"); }
    c->H = (float *)(c->ws + o_H);
    c->P = (float *)(c->ws + o_P);
    c->p_floats = p_floats;
    c->Xn = c->ws + o_Xn;
    c->Qb = c->ws + o_Qb;
    c->Ob = c->ws + o_Ob;
    c->Ab = c->ws + o_Ab;
    if (c->bf16) {
        c->Xn_lo = c->ws + o_Xl;
        c->Qb_lo = c->ws + o_Ql;
        c->Ob_lo = c->ws + o_Ol;
        c->Ab_lo = c->ws + o_Al;
    }
    c->rope_cos = (float *)(c->ws + o_cos);
    c->rope_sin = (float *)(c->ws + o_sin);
    c->attn_part = (float *)(c->ws + o_ap);
    c->d_tables = c->ws + o_tab;
    c->rs_ssq = (float *)(c->ws + o_ss);

    e = hipHostMalloc((void **)&c->h_stage, c->tables_bytes, hipHostMallocDefault);
    if (e != hipSuccess) { (void)hipFree(c->ws); delete c; return fail(nullptr, KVR_E_NOMEM, "kvr_create: pinned staging allocation failed"); }
    e = hipEventCreateWithFlags(&c->stage_ev, hipEventDisableTiming);
    if (e != hipSuccess) { (void)hipHostFree(c->h_stage); (void)hipFree(c->ws); delete c; return hip_fail(nullptr, e, "hipEventCreate"); }

    // rotary table: angles p * theta^(-2i/hd) in double precision, stored as fp32 cos/sin
    {
        const int half = hd / 2;
        std::vector<float> tc((size_t)d.max_ctx * half), ts((size_t)d.max_ctx * half);
        std::vector<double> inv(half);
        for (int i = 0; i < half; ++i) inv[i] = std::pow(d.rope_theta, -2.0 * i / (double)hd);
        for (int p = 0; p < d.max_ctx; ++p)
            for (int i = 0; i < half; ++i) {
                const double a = (double)p * inv[i];
                tc[(size_t)p * half + i] = (float)std::cos(a);
                ts[(size_t)p * half + i] = (float)std::sin(a);
            }
        e = hipMemcpy(c->rope_cos, tc.data(), tc.size() * 4, hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(c->rope_sin, ts.data(), ts.size() * 4, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipEventDestroy(c->stage_ev); (void)hipHostFree(c->h_stage); (void)hipFree(c->ws); delete c;
            return hip_fail(nullptr, e, "kvr_create: workspace initialisation");
        }
    }
    // projection weights in operand order, one contiguous copy per layer
    if (pack_ok(d, c->force_simple)) {
        const int NQKV = qd + 2 * kd;
        const size_t per_layer = (size_t)NQKV * D + (size_t)D * qd + (size_t)2 * F * D + (size_t)D * F;
        c->wpk_bytes = per_layer * 2 * d.n_layers;
        e = hipMalloc((void **)&c->wpk, c->wpk_bytes);
        if (e != hipSuccess) {
            c->wpk = nullptr;
            (void)hipEventDestroy(c->stage_ev); (void)hipHostFree(c->h_stage); (void)hipFree(c->ws); delete c;
            return fail(nullptr, KVR_E_NOMEM, "kvr_create: packed weight allocation failed");
        }
        c->pk.resize(d.n_layers);
        // gate/up tiles are stored in groups of the tile count a skinny block
        // streams (the plan for a repair of up to 64 rows), so that a block
        // reads one contiguous range: 8B shape, 48 rows, 47.8 -> 44.5 us.  The
        // tiled kernel pays 2-4 % for grouped weights (Qwen shape at 528 rows,
        // batched repair); for the other projections, which split K over
        // blocks, grouping gained the skinny path under 1 % and they stay
        // tile-major.
        const int rref = std::min(64, std::max(1, d.max_rows));
        c->gu_grp = plan_skinny(2 * F / 16, D, rref, true, 16, nullptr, nullptr).nt;
        bf16_t *dst = (bf16_t *)c->wpk;
        for (int l = 0; l < d.n_layers && e == hipSuccess; ++l) {
            const kvr_layer_weights &w = c->layers[l];
            kvr_ctx::PackedLayer &pl = c->pk[l];
            pl.qkv = dst;
            e = launch_pack_weight(w.wq, w.wk, w.wv, qd, qd + kd, false, NQKV, D, c->qkv_grp, dst, 0);
            dst += (size_t)NQKV * D;
            pl.o = dst;
            if (e == hipSuccess) e = launch_pack_weight(w.wo, w.wo, w.wo, D, D, false, D, qd, c->o_grp, dst, 0);
            dst += (size_t)D * qd;
            pl.gu = dst;
            if (e == hipSuccess)
                e = launch_pack_weight(w.w_gate, w.w_up, w.w_up, F, 2 * F, true, 2 * F, D, c->gu_grp, dst, 0);
            dst += (size_t)2 * F * D;
            pl.down = dst;
            if (e == hipSuccess) e = launch_pack_weight(w.w_down, w.w_down, w.w_down, D, D, false, D, F, c->down_grp, dst, 0);
            dst += (size_t)D * F;
        }
        if (e == hipSuccess && d.vocab % 16 == 0) {
            c->lm_pk_bytes = (size_t)d.vocab * D * 2;
            e = hipMalloc(&c->lm_pk, c->lm_pk_bytes);
            if (e == hipSuccess) e = launch_pack_weight(c->lm_head, c->lm_head, c->lm_head, d.vocab, d.vocab, false,
                                                        d.vocab, D, 1, c->lm_pk, 0);
        }
        if (e == hipSuccess) e = hipStreamSynchronize(0);
        if (e != hipSuccess) {
            if (c->lm_pk) (void)hipFree(c->lm_pk);
            (void)hipFree(c->wpk);
            (void)hipEventDestroy(c->stage_ev); (void)hipHostFree(c->h_stage); (void)hipFree(c->ws); delete c;
            return hip_fail(nullptr, e, "kvr_create: weight packing");
        }
    }
    *out = c;
    return KVR_OK;
}

void kvr_destroy(kvr_ctx *c) {
    if (!c) return;
    {
        DeviceGuard g(c->device);
        (void)hipDeviceSynchronize();
        if (c->stage_ev) (void)hipEventDestroy(c->stage_ev);
        for (auto &m : c->ev_marks) {
            (void)hipEventDestroy(m.start);
            (void)hipEventDestroy(m.stop);
        }
        for (auto ev : c->ev_pool) (void)hipEventDestroy(ev);
        if (c->h_stage) (void)hipHostFree(c->h_stage);
        if (c->ws) (void)hipFree(c->ws);
        if (c->wpk) (void)hipFree(c->wpk);
        if (c->lm_pk) (void)hipFree(c->lm_pk);
        if (c->score_y) (void)hipFree(c->score_y);
        if (c->sel_scratch) (void)hipFree(c->sel_scratch);
    }
    delete c;
}

kvr_status kvr_prefill(kvr_ctx *c, const int32_t *d_tokens, int32_t n, int32_t n_cap, void *d_cache,
                       float *d_hidden_out, void *stream) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_prefill: NULL context");
    if (!d_tokens || !d_cache) return fail(c, KVR_E_ARG, "kvr_prefill: NULL tokens or cache");
    if (!aligned16(d_cache)) return fail(c, KVR_E_ARG, "kvr_prefill: cache must be 16-byte aligned");
    if (n < 1 || n > n_cap || n_cap > c->d.max_ctx)
        return fail(c, KVR_E_RANGE, "kvr_prefill: need 1 <= n <= n_cap <= max_ctx");
    DeviceGuard g(c->device);
    hipStream_t s = (hipStream_t)stream;
    const int chunk = c->rows_cap;
    for (int c0 = 0; c0 < n; c0 += chunk) {
        const int c1 = std::min(n, c0 + chunk);
        Tables &t = c->tab;
        t.clear();
        t.docs.push_back(DocInfo{d_cache, d_tokens, d_hidden_out, n, n_cap, 0, c1 - c0});
        t.rows.reserve(c1 - c0);
        for (int p = c0; p < c1; ++p) t.rows.push_back(RowInfo{p, 0, p, 0});
        kvr_status st = run_pass(c, t, s);
        if (st != KVR_OK) return st;
    }
    return KVR_OK;
}

kvr_status kvr_transplant(kvr_ctx *c, const void *d_src, int32_t src_n_cap, void *d_dst, int32_t dst_n_cap,
                          const int32_t *h_positions, int32_t n_positions, void *stream) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_transplant: NULL context");
    if (n_positions < 0 || (n_positions > 0 && !h_positions)) return fail(c, KVR_E_ARG, "kvr_transplant: bad position list");
    if (n_positions == 0) return KVR_OK;
    if (!d_src || !d_dst) return fail(c, KVR_E_ARG, "kvr_transplant: NULL cache");
    if (!aligned16(d_src) || !aligned16(d_dst)) return fail(c, KVR_E_ARG, "kvr_transplant: caches must be 16-byte aligned");
    const int32_t lim = std::min(src_n_cap, dst_n_cap);
    for (int i = 0; i < n_positions; ++i) {
        if (h_positions[i] < 0 || h_positions[i] >= lim) return fail(c, KVR_E_RANGE, "kvr_transplant: position out of range");
        if (i > 0 && h_positions[i] <= h_positions[i - 1])
            return fail(c, KVR_E_ARG, "kvr_transplant: positions must be strictly ascending");
    }
    DeviceGuard g(c->device);
    hipStream_t s = (hipStream_t)stream;
    const size_t row = (size_t)c->d.head_dim * elem_size(c->d);
    const size_t planes = (size_t)c->d.n_layers * 2 * c->d.n_kv_heads;
    for (int i = 0; i < n_positions;) {
        int j = i + 1;
        while (j < n_positions && h_positions[j] == h_positions[j - 1] + 1) ++j;
        const size_t p0 = (size_t)h_positions[i];
        // one 2-D copy: `planes` rows of (j - i) cache rows each
        hipError_t e = hipMemcpy2DAsync((char *)d_dst + p0 * row, (size_t)dst_n_cap * row,
                                        (const char *)d_src + p0 * row, (size_t)src_n_cap * row, (size_t)(j - i) * row,
                                        planes, hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return hip_fail(c, e, "kvr_transplant: hipMemcpy2DAsync");
        i = j;
    }
    return KVR_OK;
}

kvr_status kvr_score(kvr_ctx *c, void *d_cache, int32_t n, int32_t n_cap, const int32_t *d_tokens, int32_t m,
                     float *d_logprob, int32_t *d_argmax, void *stream) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_score: NULL context");
    if (!d_cache || !d_tokens) return fail(c, KVR_E_ARG, "kvr_score: NULL cache or tokens");
    if (!aligned16(d_cache)) return fail(c, KVR_E_ARG, "kvr_score: cache must be 16-byte aligned");
    if (m > 1 && !d_logprob) return fail(c, KVR_E_ARG, "kvr_score: NULL log-probability output");
    if (n < 0 || m < 1 || (long long)n + m > n_cap || n_cap > c->d.max_ctx)
        return fail(c, KVR_E_RANGE, "kvr_score: need n >= 0, m >= 1, n + m <= n_cap <= max_ctx");
    if (m > c->rows_cap) return fail(c, KVR_E_RANGE, "kvr_score: more appended tokens than one pass holds");
    DeviceGuard g(c->device);
    kvr_status st = score_buffers(c);
    if (st != KVR_OK) return st;
    return score_block(c, d_cache, n, n_cap, d_tokens, m, d_logprob, d_argmax, nullptr, (hipStream_t)stream);
}

kvr_status kvr_generate(kvr_ctx *c, void *d_cache, int32_t n, int32_t n_cap, int32_t *d_tokens, int32_t q,
                        int32_t max_new, void *stream) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_generate: NULL context");
    if (!d_cache || !d_tokens) return fail(c, KVR_E_ARG, "kvr_generate: NULL cache or tokens");
    if (!aligned16(d_cache)) return fail(c, KVR_E_ARG, "kvr_generate: cache must be 16-byte aligned");
    if (n < 0 || q < 1 || max_new < 1 || (long long)n + q + max_new - 1 > n_cap || n_cap > c->d.max_ctx)
        return fail(c, KVR_E_RANGE, "kvr_generate: need n >= 0, q >= 1, max_new >= 1, n + q + max_new - 1 <= n_cap <= max_ctx");
    if (q > c->rows_cap) return fail(c, KVR_E_RANGE, "kvr_generate: query longer than one pass holds");
    DeviceGuard g(c->device);
    kvr_status st = score_buffers(c);
    if (st != KVR_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    // the query block, then one row per generated token; every next id is
    // written on the device and read back by the following pass
    st = score_block(c, d_cache, n, n_cap, d_tokens, q, nullptr, nullptr, d_tokens + n + q, s);
    for (int i = 1; i < max_new && st == KVR_OK; ++i)
        st = score_block(c, d_cache, n + q + i - 1, n_cap, d_tokens, 1, nullptr, nullptr, d_tokens + n + q + i, s);
    return st;
}

// Grow the selectors' scratch to at least `need` bytes (waits for the stream
// before freeing the old buffer).
static kvr_status sel_reserve(kvr_ctx *c, size_t need, hipStream_t s, const char *who) {
    if (need <= c->sel_bytes) return KVR_OK;
    if (c->sel_scratch) {
        hipError_t e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(c, e, (std::string(who) + ": hipStreamSynchronize").c_str());
        (void)hipFree(c->sel_scratch);
        c->sel_scratch = nullptr;
        c->sel_bytes = 0;
    }
    if (hipMalloc((void **)&c->sel_scratch, need) != hipSuccess)
        return fail(c, KVR_E_NOMEM, std::string(who) + ": scratch allocation failed");
    c->sel_bytes = need;
    return KVR_OK;
}

kvr_status kvr_select_cacheblend(kvr_ctx *c, const void *d_cache, int32_t n, int32_t n_cap,
                                 const int32_t *d_tokens_new, int32_t edit_start, int32_t edit_end, int32_t K,
                                 int32_t layer, int32_t *d_out, float *d_dev_out, int32_t *n_out, void *stream) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_select_cacheblend: NULL context");
    if (!d_cache || !d_tokens_new || !n_out || K < 0 || (K > 0 && !d_out))
        return fail(c, KVR_E_ARG, "kvr_select_cacheblend: NULL argument or negative K");
    if (!aligned16(d_cache)) return fail(c, KVR_E_ARG, "kvr_select_cacheblend: cache must be 16-byte aligned");
    if (n < 1 || n > n_cap || n_cap > c->d.max_ctx || edit_start < 0 || edit_start > edit_end || edit_end > n)
        return fail(c, KVR_E_RANGE, "kvr_select_cacheblend: need 1 <= n <= n_cap <= max_ctx and "
                                    "0 <= edit_start <= edit_end <= n");
    if (layer < 0 || layer >= c->d.n_layers) return fail(c, KVR_E_RANGE, "kvr_select_cacheblend: layer out of range");
    const int m = std::max(0, n - 1 - edit_end);  // pool D = [edit_end, n - 1)
    *n_out = std::min(K, m);
    if (m == 0) return KVR_OK;
    DeviceGuard g(c->device);
    hipStream_t s = (hipStream_t)stream;
    const kvr_dims &d = c->d;
    const size_t row = (size_t)d.head_dim * elem_size(d);
    const size_t cache_bytes = align_up((size_t)(layer + 1) * 2 * d.n_kv_heads * n_cap * row, 256);
    kvr_status st0 = sel_reserve(c, cache_bytes + (size_t)n_cap * 4, s, "kvr_select_cacheblend");
    if (st0 != KVR_OK) return st0;
    char *work = c->sel_scratch;  // scratch cache copy, then the deviations
    float *dev = d_dev_out ? d_dev_out : (float *)(work + cache_bytes);
    // layers below `layer`, positions before the edit: the stale states (the
    // edit does not reach them) for the suffix forward to attend over
    if (layer > 0 && edit_start > 0) {
        hipError_t e = hipMemcpy2DAsync(work, (size_t)n_cap * row, d_cache, (size_t)n_cap * row,
                                        (size_t)edit_start * row, (size_t)layer * 2 * d.n_kv_heads,
                                        hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return hip_fail(c, e, "kvr_select_cacheblend: hipMemcpy2DAsync");
    }
    // the suffix [edit_start, n) of C' through layers 0..layer-1 and the
    // key/value projection of `layer`, into the work cache
    for (int c0 = edit_start; c0 < n; c0 += c->rows_cap) {
        const int c1 = std::min(n, c0 + c->rows_cap);
        Tables &t = c->tab;
        t.clear();
        t.docs.push_back(DocInfo{work, d_tokens_new, nullptr, n, n_cap, 0, c1 - c0});
        t.rows.reserve(c1 - c0);
        for (int p = c0; p < c1; ++p) t.rows.push_back(RowInfo{p, 0, p - c0, 0});
        kvr_status st = run_pass(c, t, s, layer);
        if (st != KVR_OK) return st;
    }
    hipError_t e = launch_kv_deviation(c->bf16, work, n_cap, layer, d_cache, n_cap, layer, d.n_kv_heads,
                                       d.head_dim, edit_end, n - 1, dev, s);
    if (e == hipSuccess) e = launch_topk(dev, m, *n_out, edit_end, d_out, s);
    if (e != hipSuccess) return hip_fail(c, e, "kvr_select_cacheblend: deviation / top-K");
    return KVR_OK;
}

// Shared body of the two Attention-selector entry points.  `buf` null: the
// scratch comes from the context (grown on demand); otherwise `buf` holds
// `cap` bytes of device scratch and nothing is allocated.
static kvr_status select_attention(kvr_ctx *c, const char *who, void *d_cache, int32_t n, int32_t n_cap,
                                   const int32_t *d_tokens, int32_t q, int32_t edit_start, int32_t edit_end,
                                   int32_t K, int32_t *d_out, float *d_mass_out, int32_t *n_out, void *stream,
                                   char *buf, size_t cap) {
    if (!c) return fail(nullptr, KVR_E_ARG, std::string(who) + ": NULL context");
    if (!d_cache || !d_tokens || !n_out || K < 0 || (K > 0 && !d_out))
        return fail(c, KVR_E_ARG, std::string(who) + ": NULL argument or negative K");
    if (!aligned16(d_cache)) return fail(c, KVR_E_ARG, std::string(who) + ": cache must be 16-byte aligned");
    if (n < 1 || q < 1 || (long long)n + q > n_cap || n_cap > c->d.max_ctx || edit_start < 0 ||
        edit_start > edit_end || edit_end > n)
        return fail(c, KVR_E_RANGE, std::string(who) + ": need 1 <= n, 1 <= q, n + q <= n_cap <= max_ctx and "
                                                       "0 <= edit_start <= edit_end <= n");
    if (q > c->rows_cap) return fail(c, KVR_E_RANGE, std::string(who) + ": query longer than one pass holds");
    const kvr_dims &d = c->d;
    const size_t part_bytes = align_up((size_t)d.n_kv_heads * n * 4, 256);
    const size_t lse_bytes = align_up((size_t)q * d.n_heads * 4, 256);
    const size_t need = part_bytes + lse_bytes + (d_mass_out ? 0 : (size_t)n * 4);
    if (buf && need > cap)
        return fail(c, KVR_E_RANGE, std::string(who) + ": needs " + std::to_string(need) +
                                        " bytes of scratch, more than the fixed " + std::to_string(cap));
    const int m = std::max(0, n - 1 - edit_end);  // pool D = [edit_end, n - 1)
    *n_out = std::min(K, m);
    if (m == 0 && !d_mass_out) return KVR_OK;
    DeviceGuard g(c->device);
    hipStream_t s = (hipStream_t)stream;
    if (!buf) {
        kvr_status st = sel_reserve(c, need, s, who);
        if (st != KVR_OK) return st;
        buf = c->sel_scratch;
    }
    // part [Hkv][n] is written (not accumulated) at layer 0 and lse at every
    // layer before it is read, so the scratch needs no clearing
    MassHook mh{d_cache, n_cap, n, (float *)(buf + part_bytes), (float *)buf};
    float *mass = d_mass_out ? d_mass_out : (float *)(buf + part_bytes + lse_bytes);
    // the query rows at positions [n, n + q) over the stale cache (their own
    // keys/values land in slots [n, n + q))
    Tables &t = c->tab;
    t.clear();
    t.docs.push_back(DocInfo{d_cache, d_tokens, nullptr, n + q, n_cap, 0, q});
    for (int j = 0; j < q; ++j) t.rows.push_back(RowInfo{n + j, 0, j, 0});
    kvr_status st = run_pass(c, t, s, -1, &mh);
    if (st != KVR_OK) return st;
    hipError_t e = launch_mass_reduce(mh.part, d.n_kv_heads, n, mass, s);
    if (e == hipSuccess && m > 0) e = launch_topk(mass + edit_end, m, *n_out, edit_end, d_out, s);
    if (e != hipSuccess) return hip_fail(c, e, (std::string(who) + ": reduce / top-K").c_str());
    return KVR_OK;
}

kvr_status kvr_select_attention(kvr_ctx *c, void *d_cache, int32_t n, int32_t n_cap, const int32_t *d_tokens,
                                int32_t q, int32_t edit_start, int32_t edit_end, int32_t K, int32_t *d_out,
                                float *d_mass_out, int32_t *n_out, void *stream) {
    return select_attention(c, "kvr_select_attention", d_cache, n, n_cap, d_tokens, q, edit_start, edit_end, K,
                            d_out, d_mass_out, n_out, stream, nullptr, 0);
}

kvr_status kvr_select_attention_noalloc(kvr_ctx *c, void *d_cache, int32_t n, int32_t n_cap,
                                        const int32_t *d_tokens, int32_t q, int32_t edit_start, int32_t edit_end,
                                        int32_t K, int32_t *d_out, float *d_mass_out, int32_t *n_out, void *stream) {
    if (c && !c->scratch_ptr)
        return fail(c, KVR_E_HIP, std::string("kvr_select_attention_noalloc: the device scratch has no address (") +
                                      hipGetErrorString(c->scratch_err) + ")");
    return select_attention(c, "kvr_select_attention_noalloc", d_cache, n, n_cap, d_tokens, q, edit_start, edit_end,
                            K, d_out, d_mass_out, n_out, stream, (char *)(c ? c->scratch_ptr : nullptr),
                            NOALLOC_SCRATCH_BYTES);
}

kvr_status kvr_profile_enable(kvr_ctx *c, int32_t enable) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_profile_enable: NULL context");
    c->profiling = enable != 0;
    return KVR_OK;
}

kvr_status kvr_profile_read(kvr_ctx *c, int32_t capacity, const char **names, double *total_ms, int64_t *launches,
                            int32_t *n_steps) {
    if (!c || !n_steps || capacity < 0 || (capacity > 0 && (!names || !total_ms || !launches)))
        return fail(c, KVR_E_ARG, "kvr_profile_read: bad arguments");
    DeviceGuard g(c->device);
    if (!c->ev_marks.empty()) {
        hipError_t e = hipEventSynchronize(c->ev_marks.back().stop);
        if (e != hipSuccess) return hip_fail(c, e, "kvr_profile_read");
        for (const auto &m : c->ev_marks) {
            float ms = 0.f;
            e = hipEventElapsedTime(&ms, m.start, m.stop);
            if (e != hipSuccess) return hip_fail(c, e, "kvr_profile_read: hipEventElapsedTime");
            c->step_ms[m.step] += ms;
            c->step_n[m.step] += 1;
        }
        for (const auto &m : c->ev_marks) {
            c->ev_pool.push_back(m.start);
            c->ev_pool.push_back(m.stop);
        }
        c->ev_marks.clear();
    }
    *n_steps = ST_COUNT;
    for (int i = 0; i < ST_COUNT && i < capacity; ++i) {
        names[i] = STEP_NAMES[i];
        total_ms[i] = c->step_ms[i];
        launches[i] = c->step_n[i];
    }
    for (int i = 0; i < ST_COUNT; ++i) { c->step_ms[i] = 0.0; c->step_n[i] = 0; }
    return KVR_OK;
}

kvr_status kvr_repair(kvr_ctx *c, const kvr_doc *docs, int32_t n_docs, void *stream) {
    if (!c) return fail(nullptr, KVR_E_ARG, "kvr_repair: NULL context");
    if (n_docs < 0 || (n_docs > 0 && !docs)) return fail(c, KVR_E_ARG, "kvr_repair: bad document array");
    long long total = 0;
    for (int i = 0; i < n_docs; ++i) {
        const kvr_doc &dc = docs[i];
        const std::string tag = "kvr_repair: document " + std::to_string(i) + ": ";
        if (dc.n_positions < 0 || (dc.n_positions > 0 && !dc.h_positions))
            return fail(c, KVR_E_ARG, tag + "bad position list");
        if (dc.n < 1 || dc.n > dc.n_cap || dc.n_cap > c->d.max_ctx)
            return fail(c, KVR_E_RANGE, tag + "need 1 <= n <= n_cap <= max_ctx");
        if (dc.edit_start < 0 || dc.edit_start > dc.edit_end || dc.edit_end > dc.n)
            return fail(c, KVR_E_RANGE, tag + "need 0 <= edit_start <= edit_end <= n");
        for (int j = 0; j < dc.n_positions; ++j) {
            const int p = dc.h_positions[j];
            if (p < 0 || p >= dc.n) return fail(c, KVR_E_RANGE, tag + "position outside [0, n)");
            if (j > 0 && p <= dc.h_positions[j - 1])
                return fail(c, KVR_E_ARG, tag + "positions must be strictly ascending");
            if (p >= dc.edit_start && p < dc.edit_end) return fail(c, KVR_E_ARG, tag + "position inside the edit span");
        }
        const long long np = (long long)(dc.edit_end - dc.edit_start) + dc.n_positions;
        if (np > 0 && (!dc.d_cache || !dc.d_tokens_new)) return fail(c, KVR_E_ARG, tag + "NULL cache or tokens");
        if (np > 0 && !aligned16(dc.d_cache)) return fail(c, KVR_E_ARG, tag + "cache must be 16-byte aligned");
        total += np;
    }
    if (total > c->d.max_rows) return fail(c, KVR_E_RANGE, "kvr_repair: total |P| exceeds max_rows");
    if (total == 0) return KVR_OK;
    // Documents of one call are repaired in one pass: every document's fresh
    // rows of a layer are scattered before any row attends.  Two documents
    // sharing cache memory would then read each other's fresh rows, which two
    // separate repairs would not, so overlapping caches are rejected.
    {
        std::vector<std::pair<uintptr_t, uintptr_t>> spans;
        for (int i = 0; i < n_docs; ++i) {
            const kvr_doc &dc = docs[i];
            if ((dc.edit_end - dc.edit_start) + dc.n_positions == 0) continue;
            const uintptr_t b = (uintptr_t)dc.d_cache;
            spans.push_back({b, b + kvr_cache_bytes(&c->d, dc.n_cap)});
        }
        std::sort(spans.begin(), spans.end());
        for (size_t i = 1; i < spans.size(); ++i)
            if (spans[i].first < spans[i - 1].second)
                return fail(c, KVR_E_ARG, "kvr_repair: two documents share cache memory");
    }

    Tables &t = c->tab;
    t.clear();
    t.rows.reserve((size_t)total);
    for (int i = 0; i < n_docs; ++i) {
        const kvr_doc &dc = docs[i];
        const int np = (dc.edit_end - dc.edit_start) + dc.n_positions;
        if (np == 0) continue;
        const int di = (int)t.docs.size();
        t.docs.push_back(DocInfo{dc.d_cache, dc.d_tokens_new, dc.d_hidden_out, dc.n, dc.n_cap, (int)t.rows.size(), np});
        // merge the span and the (sorted, disjoint) positions in ascending order
        int j = 0, out = 0;
        for (int p = dc.edit_start; p <= dc.edit_end; ++p) {
            while (j < dc.n_positions && dc.h_positions[j] < p) t.rows.push_back(RowInfo{dc.h_positions[j++], di, out++, 0});
            if (p < dc.edit_end) t.rows.push_back(RowInfo{p, di, out++, 0});
        }
        while (j < dc.n_positions) t.rows.push_back(RowInfo{dc.h_positions[j++], di, out++, 0});
    }
    DeviceGuard g(c->device);
    return run_pass(c, t, (hipStream_t)stream);
}

}  // extern "C"
