// Host side of libasv: argument checks, workspace layouts, tile selection and the launch
// sequences of one verification step, one draft step, the pruning of the draft trees, the
// tree-attention metadata and the commit. Every entry point is declared in include/asv.h.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include <cstdio>

#include "asv.h"
#include "k_accept.h"
#include "k_draft.h"
#include "k_lmhead.h"
#include "k_reduce.h"
#include "k_tree.h"

namespace asv {
namespace {

constexpr size_t kAlign = 256;

// Vocabulary rows per K1 workgroup tile = width of one record slab; every tile family below
// uses this width, so the record layout depends only on V.
constexpr int kSlab = 256;
constexpr int kPackRowsTarget = 256;   // rows per tile of the packed target LM-head weight
constexpr int kPackRowsDraft = 64;     // rows per tile of the packed draft LM-head weight

// Text of the most recent failure on this host thread (see asv_last_error).
thread_local char g_last_error[256] = "";

void set_error(const char* what, hipError_t e) {
  snprintf(g_last_error, sizeof(g_last_error), "%s: %s (%d)", what, hipGetErrorString(e),
           (int)e);
}

// ASV_OK when the launches enqueued so far succeeded, else ASV_EHIP with the error recorded.
int launch_status(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return ASV_OK;
  set_error(what, e);
  return ASV_EHIP;
}

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Tile families of K1. Few rows (the weight-streaming regime of small batches) use a 64-row
// tile so that all rows share one pass over W. Beyond 64 rows the plan minimises an estimate of
// the time: the rounds of workgroups over the CUs times the time of one tile, 62 : 80 : 98 for
// the 128-, 192- and 256-row tiles (per-round times of the spread loops on MI355X, with the
// packed weight); ties go to the larger tile. Interleaved comparisons at V = 151936 (records
// bit-identical across the tiles) agree with the single-family estimate at every row count
// measured from 150 to 3048 rows: e.g. at 540 rows three 192-row tiles beat three 256-row tiles
// by 17%, at 700 rows three 256-row tiles beat four 192-row tiles by 9%.
// A plan may split the slabs between two families in two launches: the first n1 slabs on
// family a, the rest on family b, n1 chosen so that family a fills whole rounds. At 378 rows
// and V = 151936, for instance, one 192-row family takes 1188 tiles, 4.64 rounds run as 5;
// 128-row tiles on 85 slabs (255 tiles, one round) and 192-row tiles on the other 509 (1018
// tiles, four rounds) leave no round a third empty.
enum class Tile { kRows64, kRows128, kRows192, kRows256 };

struct K1Plan {
  Tile a, b;       // slabs [0, n1) on tile a, [n1, S) on tile b
  int n1;          // == S: one launch of tile a
};


// Compute units of the current device, queried once per device.
int cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

K1Plan plan_k1(int N, int S, int cus) {
  if (N <= 64) return K1Plan{Tile::kRows64, Tile::kRows64, S};
  struct Family { Tile tile; int rows; int cost; };
  const Family families[3] = {{Tile::kRows128, 128, 62}, {Tile::kRows192, 192, 80},
                              {Tile::kRows256, 256, 98}};
  auto rounds = [&](int64_t tiles) { return (tiles + cus - 1) / cus; };
  K1Plan best{Tile::kRows128, Tile::kRows128, S};
  int64_t best_est = INT64_MAX;
  for (const Family& f : families) {
    const int64_t est = rounds((int64_t)((N + f.rows - 1) / f.rows) * S) * f.cost;
    if (est <= best_est) {
      best_est = est;
      best = K1Plan{f.tile, f.tile, S};
    }
  }
  // two families: family a fills k whole rounds on its slabs, family b takes the rest; taken
  // only when strictly better than every single family. The search stops at kMaxSplitRounds
  // rounds of family a (a launch that long gains nothing from a finer split, and the bound
  // keeps the host loop short for any size the checks accept).
  constexpr int64_t kMaxSplitRounds = 4096;
  for (const Family& fa : families) {
    const int64_t ra = (N + fa.rows - 1) / fa.rows;
    for (const Family& fb : families) {
      if (fb.rows == fa.rows) continue;
      const int64_t rb = (N + fb.rows - 1) / fb.rows;
      for (int64_t k = 1; k <= kMaxSplitRounds && k * cus < (int64_t)S * ra; ++k) {
        const int64_t n1 = k * cus / ra;
        if (n1 <= 0 || n1 >= S) continue;
        const int64_t est = rounds(n1 * ra) * fa.cost + rounds((S - n1) * rb) * fb.cost;
        if (est < best_est) {
          best_est = est;
          best = K1Plan{fa.tile, fb.tile, (int)n1};
        }
      }
    }
  }
  return best;
}

// Order of a K1 launch's tiles. The blocks are dealt to the 8 XCDs in contiguous runs, and the
// concurrent tiles of an XCD (cus / 8 of them) share what they read through its L2: in the
// slab-major order about c / RT W slabs and all RT X row tiles per round of c tiles, blocked
// into groups of 4 row tiles, c / 4 slabs and 4 row tiles. Per round an XCD then reads about
// c / RT + RT or c / 4 + 4 slabs' and row tiles' worth of data from beyond its L2; the blocked
// order is taken where it reads less (at 256 CUs: more than 8 row tiles). Measured at 3048
// rows (12 row tiles): K1 1.3-1.6% faster, with blocks of 8 slabs x 4 row tiles.
void tile_blocking(int RT, int cus, int* blk_slabs, int* blk_rows) {
  constexpr int kRows = 4;
  const int c = std::max(1, cus / 8);
  *blk_slabs = 0;
  *blk_rows = 0;
  if (RT > kRows && (double)c / RT + RT > (double)c / kRows + kRows) {
    *blk_slabs = std::max(1, c / kRows);
    *blk_rows = kRows;
  }
}

// Whether a launch of `tiles` 64-row tiles runs the one-slot ring: its workgroups fit three
// per CU but not two. Same-box A/Bs (K1, up to 64 rows): at V = 151936 (594 tiles on 256
// CUs) 5.3% faster at 60 rows and 2.2% at 30; outside this range it was slower (V = 64000,
// 250 tiles: +7%; V = 200000, 782 tiles: +6%) or level (V = 128256, 501 tiles).
bool one_slot_64(int tiles, int cus) { return tiles > 2 * cus && tiles <= 3 * cus; }

// Launches of at most this many row tiles copy W with the non-temporal hint (the one or two
// tiles of a slab read it about once); more row tiles share each W slab through an XCD's L2
// and keep the default policy. Against the earlier rule (the hint for tiles of up to 128 rows)
// in same-box A/Bs: 260, 300, 378 and 450 rows 3% faster, 150 rows 1.4%, 500 rows 1%; 128,
// 200 and 600 to 3048 rows level.
constexpr int kStreamWMaxRowTiles = 2;

int tile_rows_of(Tile t) {
  switch (t) {
    case Tile::kRows64: return 64;
    case Tile::kRows128: return 128;
    case Tile::kRows192: return 192;
    default: return 256;
  }
}

// The K1 launches of a verification step over N rows and S slabs on `cus` CUs: the plan's one
// or two launches, each with its K loop, W copy policy and tile order. Returns the count.
int k1_launches(int N, int S, int cus, const K1Plan& plan, asv_k1_launch out[2]) {
  int n = 0;
  auto add = [&](Tile t, int slab0, int n_slabs) {
    asv_k1_launch& k = out[n++];
    k.tile_rows = tile_rows_of(t);
    k.slab0 = slab0;
    k.n_slabs = n_slabs;
    k.row_tiles = (N + k.tile_rows - 1) / k.tile_rows;
    const int tiles = n_slabs * k.row_tiles;
    switch (t) {
      case Tile::kRows64: k.k_loop = one_slot_64(tiles, cus) ? 1 : 0; break;
      case Tile::kRows128: k.k_loop = 3; break;
      default: k.k_loop = 2; break;
    }
    k.stream_w = k.row_tiles <= kStreamWMaxRowTiles ? 1 : 0;
    tile_blocking(k.row_tiles, cus, &k.blk_slabs, &k.blk_rows);
  };
  add(plan.a, 0, plan.n1);
  if (plan.n1 < S) add(plan.b, plan.n1, S - plan.n1);
  return n;
}

// The tile asv_verify_args.k1_tile_rows asks for; false for a value that names no tile.
bool forced_tile(int rows, Tile* t) {
  switch (rows) {
    case 64: *t = Tile::kRows64; return true;
    case 128: *t = Tile::kRows128; return true;
    case 192: *t = Tile::kRows192; return true;
    case 256: *t = Tile::kRows256; return true;
    default: return false;
  }
}

struct Layout {
  int S = 0;       // vocabulary slabs
  int n_conf = 0;  // draft-confidence chunks per request
  size_t off_rec_m = 0, off_rec_s = 0, off_rec_a = 0, off_conf_m = 0, off_conf_s = 0;
  size_t off_cnt = 0;  // B + 1 ints: per-request completion counters, then the bad-offsets flag
  size_t bytes = 0;
};

Layout layout(int B, int N, int V) {
  Layout L;
  L.S = (V + kSlab - 1) / kSlab;
  L.n_conf = (V + kConfChunk - 1) / kConfChunk;
  const size_t rec = (size_t)N * L.S * 4;
  const size_t conf = (size_t)B * L.n_conf * 4;
  size_t at = 0;
  L.off_rec_m = at;  at += align_up(rec);
  L.off_rec_s = at;  at += align_up(rec);
  L.off_rec_a = at;  at += align_up(rec);
  L.off_conf_m = at; at += align_up(conf);
  L.off_conf_s = at; at += align_up(conf);
  L.off_cnt = at;    at += align_up((size_t)(B + 1) * 4);
  L.bytes = at;
  return L;
}

// Row and vocabulary indices (rounded up to whole tiles) and the LM-head kernel's workgroup
// count stay ints: N, V < 2^30, and for the 64-row tile, which has the most workgroups,
// ceil(V / 256) * ceil(N / 64) < 2^31.
bool grid_ok(int N, int V) {
  if (N >= (1 << 30) || V >= (1 << 30)) return false;
  const int64_t S = ((int64_t)V + kSlab - 1) / kSlab, RT = ((int64_t)N + 63) / 64;
  return S * RT < ((int64_t)1 << 31);
}

bool sizes_ok(int B, int N, int H, int V) {
  if (B < 0 || N < 0 || H <= 0 || V <= 0) return false;
  if ((B == 0) != (N == 0) || N < B) return false;
  if (H % kKAlign != 0 || H > (1 << 20)) return false;
  return grid_ok(N, V);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool params_ok(const asv_params& p) {
  if (!(p.alpha > 0.f && p.alpha <= 1.f) || p.breaker_n < 1 || p.max_promotions < -1)
    return false;
  if (!(p.dcs_divisor > 0.f && p.dcs_divisor < __builtin_inff())) return false;
  if (!(p.temperature > 0.f && p.temperature < __builtin_inff())) return false;
  for (int k = 0; k < 3; ++k)
    if (p.shape_lo[k] < 1 || p.shape_hi[k] < 1 || p.shape_start[k] < 1) return false;
  return true;
}

// K1 over the vocabulary slabs [slab0, slab0 + n_slabs).
// Launches `kernel` on `s`; with a start or stop event (measurement only) through
// hipExtLaunchKernelGGL, which sets the events to the dispatch's own start and end times.
template <typename F, typename... Args>
void launch_timed(F kernel, int grid, int threads, hipStream_t s, hipEvent_t start,
                  hipEvent_t stop, Args... args) {
  if (start || stop)
    hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(threads), 0, s, start, stop, 0, args...);
  else
    kernel<<<grid, threads, 0, s>>>(args...);
}

template <int TV, int TR, int WV, int WR, int BK, int NST, int LOOP>
void launch_lmhead(const asv_verify_args* a, const Layout& L, char* ws, hipStream_t s,
                   const asv_k1_launch& k, hipEvent_t start, hipEvent_t stop) {
  static_assert(TV == kSlab, "tiles span exactly one record slab");
  static_assert(TV == kPackRowsTarget && BK == kPackDepth, "a stage is one packed tile");
  const int grid = k.n_slabs * k.row_tiles;
  auto go = [&](auto kernel) {
    launch_timed(kernel, grid, WV * WR * kWave, s, start, stop, a->hidden, a->w_lm, a->parent,
                 a->draft_tok, a->req_offsets, a->B, a->N, a->H, a->V, L.S, k.slab0,
                 k.row_tiles, reinterpret_cast<float*>(ws + L.off_rec_m),
                 reinterpret_cast<float*>(ws + L.off_rec_s),
                 reinterpret_cast<int32_t*>(ws + L.off_rec_a), a->drafted_logit,
                 reinterpret_cast<int32_t*>(ws + L.off_cnt), a->B + 1,
                 a->w_lm_layout == ASV_W_PACKED ? 1 : 0, k.blk_slabs, k.blk_rows);
  };
  if (k.stream_w)
    go(k_lmhead_partial<TV, TR, WV, WR, BK, NST, LOOP, true>);
  else
    go(k_lmhead_partial<TV, TR, WV, WR, BK, NST, LOOP, false>);
}

// Total bytes of the packed copy of a [V][H] weight whose K blocks hold V rounded up to
// `align` rows; false for sizes the LM-head kernels reject and for copies of 4 GiB or more,
// past the 32-bit offsets they use in it.
bool packed_size(int V, int H, int align, uint64_t* bytes) {
  if (V <= 0 || H <= 0 || H % kPackDepth != 0 || H > (1 << 20)) return false;
  const uint64_t Vp = ((uint64_t)V + align - 1) / align * align;
  const uint64_t total = Vp * (uint64_t)H * 2;
  if (total >= ((uint64_t)1 << 32)) return false;
  *bytes = total;
  return true;
}

// Pack w into tiles of PR rows (k_pack_tiles), after the checks both pack entry points share.
template <int PR>
int pack_tiles(const uint16_t* w, int V, int H, uint16_t* packed, uint64_t packed_bytes,
               void* stream) {
  constexpr int kAlign = PR > 128 ? PR : 128;
  uint64_t need = 0;
  if (!packed_size(V, H, kAlign, &need) || !w || !packed || !aligned16(w) ||
      !aligned16(packed) || packed_bytes < need)
    return ASV_EINVAL;
  const uintptr_t w0 = reinterpret_cast<uintptr_t>(w), p0 = reinterpret_cast<uintptr_t>(packed);
  if (w0 < p0 + need && p0 < w0 + (uint64_t)V * H * 2) return ASV_EINVAL;   // overlap
  (void)hipGetLastError();
  const int T = (int)((need / 2 / H) / PR);        // tiles per 64-column block
  const int tiles = T * (H / kPackDepth);
  k_pack_tiles<PR><<<tiles, kPackThreads, 0, reinterpret_cast<hipStream_t>(stream)>>>(
      reinterpret_cast<const uint4*>(w), reinterpret_cast<uint4*>(packed), V, H, T);
  return launch_status("k_pack_tiles");
}

AcceptArgs accept_args(const asv_verify_args* a, const Layout& L, char* ws, bool conf) {
  AcceptArgs r;
  r.B = a->B;
  r.N = a->N;
  r.V = a->V;
  r.off = a->req_offsets;
  r.parent = a->parent;
  r.tok = a->draft_tok;
  r.tau = a->tau;
  r.row_max = a->row_max;
  r.row_arg = a->row_argmax;
  r.g = a->drafted_logit;
  r.accept = a->accept;
  r.acc_len = a->accepted_len;
  r.bonus = a->bonus_token;
  r.path = a->accepted_path;
  r.conf_m = reinterpret_cast<const float*>(ws + L.off_conf_m);
  r.conf_s = reinterpret_cast<const float*>(ws + L.off_conf_s);
  r.n_conf = conf ? L.n_conf : 0;
  r.draft_conf = a->draft_conf;
  r.state = a->state;
  r.status = a->req_status;
  r.prm = a->params;
  return r;
}

// ---- draft side

// Tile families of the draft LM head (K5), by draft rows R = 4B. The draft vocabulary is small
// (tens of thousands of rows), so narrow vocabulary slabs keep the launch above the CU count.
// Beyond 64 rows the 128-row tile repeats over row tiles (a 256-row tile with the top-4
// epilogue exceeds the register file).
enum class DraftTile { kRows32, kRows64, kRows128 };

DraftTile pick_draft_tile(int R) {
  if (R <= 32) return DraftTile::kRows32;
  if (R <= 64) return DraftTile::kRows64;
  return DraftTile::kRows128;
}

int draft_slab(DraftTile t) { return t == DraftTile::kRows128 ? 128 : 64; }

struct DraftLayout {
  int S = 0;  // vocabulary slabs of the chosen tile
  size_t off_k = 0, off_s = 0, bytes = 0;
};

DraftLayout draft_layout(int B, int V) {
  DraftLayout L;
  const int R = B * kTopK;
  L.S = (V + draft_slab(pick_draft_tile(R)) - 1) / draft_slab(pick_draft_tile(R));
  const size_t rec = (size_t)R * L.S;
  size_t at = 0;
  L.off_k = at; at += align_up(rec * kTopK * 8);
  L.off_s = at; at += align_up(rec * 4);
  L.bytes = at;
  return L;
}

bool draft_sizes_ok(int B, int H, int V) {
  if (B < 0 || H <= 0 || V < kTopK || V >= (1 << 30)) return false;
  if (H % kKAlign != 0 || H > (1 << 20)) return false;
  // 32-bit offsets inside a tile's buffer resource: all 4B rows of X and one slab of W
  if ((int64_t)B * kTopK * H * 2 >= (int64_t)1 << 31) return false;
  // the draft LM head's workgroup count stays an int
  const int R = B * kTopK;
  const DraftTile t = pick_draft_tile(R);
  const int tr = t == DraftTile::kRows32 ? 32 : t == DraftTile::kRows64 ? 64 : 128;
  const int64_t S = ((int64_t)V + draft_slab(t) - 1) / draft_slab(t);
  return S * (((int64_t)R + tr - 1) / tr) < ((int64_t)1 << 31);
}

template <int TV, int TR, int WV, int WR, int BK, int NST>
void launch_draft(const asv_draft_args* a, const DraftLayout& L, char* ws, hipStream_t s,
                  hipEvent_t start, hipEvent_t stop) {
  static_assert(BK == kPackDepth && TV % kPackRowsDraft == 0 && 128 % TV == 0,
                "a stage is one or two consecutive packed draft tiles");
  const int R = a->B * kTopK;
  const int RT = (R + TR - 1) / TR;
  launch_timed(k_draft_partial<TV, TR, WV, WR, BK, NST>, L.S * RT, WV * WR * kWave, s, start, stop,
      a->hidden, a->w_draft, R, a->H, a->V, L.S, RT, reinterpret_cast<uint64_t*>(ws + L.off_k),
      reinterpret_cast<float*>(ws + L.off_s), a->w_draft_layout == ASV_W_PACKED ? 1 : 0);
}

// ---- static scratch of asv_verify_noalloc

// The workspace of asv_verify_noalloc. In host code `scratch` names a host-side stand-in, not
// the device array: the device address comes from hipGetSymbolAddress, once per device (each
// GPU holds its own copy at its own address).
__device__ __align__(256) char scratch[ASV_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device, or nullptr (error recorded).
void* scratch_address() {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_error("hipGetDevice", e);
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("asv_verify_noalloc: device ordinal out of range", hipErrorInvalidDevice);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error("hipGetSymbolAddress(scratch)", e != hipSuccess ? e : hipErrorInvalidSymbol);
      return nullptr;
    }
    addr[dev] = p;
  }
  return addr[dev];
}

}  // namespace
}  // namespace asv

using namespace asv;

extern "C" int asv_version(void) { return ASV_VERSION; }

extern "C" const char* asv_last_error(void) { return g_last_error; }

extern "C" const char* asv_status_string(int code) {
  switch (code) {
    case ASV_OK: return "ok";
    case ASV_EINVAL: return "invalid argument (size, null or misaligned pointer, parameter)";
    case ASV_EWORKSPACE: return "workspace too small or not 256-byte aligned";
    case ASV_EHIP: return "HIP runtime error or kernel launch failure";
    case ASV_ESCRATCH:
      return "the sizes need more workspace than the static scratch of asv_verify_noalloc";
    default: return "unknown asv status code";
  }
}

extern "C" int asv_workspace_bytes(int32_t B, int32_t N, int32_t H, int32_t V,
                                   uint64_t* bytes) {
  if (!bytes || !sizes_ok(B, N, H, V)) return ASV_EINVAL;
  *bytes = layout(B, N, V).bytes;
  return ASV_OK;
}

extern "C" int asv_state_init(asv_req_state* state, int32_t B, const asv_params* p,
                              void* stream) {
  if (B < 0 || !p || (B > 0 && !state) || !params_ok(*p)) return ASV_EINVAL;
  if (B == 0) return ASV_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  k_state_init<<<(B + 255) / 256, 256, 0, s>>>(state, B, *p);
  return launch_status("k_state_init");
}

extern "C" int asv_tree_policy(const float* conf, asv_req_state* state, int32_t B,
                               const asv_params* p, void* stream) {
  if (B < 0 || !p || (B > 0 && !state) || !params_ok(*p)) return ASV_EINVAL;
  if (B == 0) return ASV_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  k_tree_policy<<<(B + 255) / 256, 256, 0, s>>>(conf, state, B, *p);
  return launch_status("k_tree_policy");
}

extern "C" int asv_verify_tuned(const asv_verify_args* a, const asv_tuning* tuning,
                                void* workspace, uint64_t workspace_bytes, void* stream) {
  if (!a || !sizes_ok(a->B, a->N, a->H, a->V)) return ASV_EINVAL;
  const asv_tuning tu = tuning ? *tuning : asv_tuning{nullptr, nullptr, 0};
  Tile forced = Tile::kRows64;
  if (tu.tile_rows != 0 && !forced_tile(tu.tile_rows, &forced)) return ASV_EINVAL;
  if (a->w_lm_layout != ASV_W_ROW_MAJOR && a->w_lm_layout != ASV_W_PACKED) return ASV_EINVAL;
  uint64_t packed_bytes = 0;
  if (a->w_lm_layout == ASV_W_PACKED &&
      !packed_size(a->V, a->H, kPackRowsTarget, &packed_bytes))
    return ASV_EINVAL;
  if (a->B == 0) return ASV_OK;
  if (!a->hidden || !a->w_lm || !a->draft_tok || !a->parent || !a->req_offsets || !a->tau ||
      !a->row_max || !a->row_lse || !a->row_argmax || !a->drafted_logit || !a->accept ||
      !a->accepted_len || !a->bonus_token || !a->accepted_path || !a->req_status)
    return ASV_EINVAL;
  if (!aligned16(a->hidden) || !aligned16(a->w_lm)) return ASV_EINVAL;
  if (!params_ok(a->params)) return ASV_EINVAL;
  const Layout L = layout(a->B, a->N, a->V);
  if (!workspace || workspace_bytes < L.bytes ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return ASV_EWORKSPACE;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  const bool conf = a->draft_logits != nullptr;
  (void)hipGetLastError();

  // K4 first: it only needs the inputs and overlaps nothing it depends on.
  if (conf) {
    k_draft_conf_partial<<<dim3(L.n_conf, a->B), kConfThreads, 0, s>>>(
        a->N, a->V, a->req_offsets, a->draft_logits, reinterpret_cast<float*>(ws + L.off_conf_m),
        reinterpret_cast<float*>(ws + L.off_conf_s));
    if (int rc = launch_status("k_draft_conf_partial")) return rc;
  }

  const K1Plan plan = tu.tile_rows != 0 ? K1Plan{forced, forced, L.S}
                                         : plan_k1(a->N, L.S, cu_count());
  asv_k1_launch k1[2];
  const int n_k1 = k1_launches(a->N, L.S, cu_count(), plan, k1);
  // timing events (measurement only): the start of the first launch, the end of the last
  const hipEvent_t ev_begin = reinterpret_cast<hipEvent_t>(tu.begin_event);
  const hipEvent_t ev_end = reinterpret_cast<hipEvent_t>(tu.end_event);
  for (int q = 0; q < n_k1; ++q) {
    const asv_k1_launch& k = k1[q];
    const hipEvent_t start = q == 0 ? ev_begin : nullptr;
    const hipEvent_t stop = q == n_k1 - 1 ? ev_end : nullptr;
    // <vocab rows, tree rows, waves along vocab, waves along rows, K per stage, ring depth,
    // K loop>, each the fastest of a sweep on MI355X for its row range. The weight-streaming
    // 64-row tile keeps two workgroups per CU (80 KB of LDS each) with the burst ring, or
    // three (40 KB each) with the one-slot ring when that takes every tile at once; a 3-deep
    // ring with one workgroup per CU was 0.7% slower in an interleaved comparison over ten
    // placements of W. The 128-, 192- and 256-row tiles run the spread K loops (copies spaced
    // between the MFMAs), in interleaved comparisons 28% faster than the burst ring at 378
    // rows and 20% at 2048 and 3048 rows.
    switch (k.tile_rows) {
      case 64:
        if (k.k_loop == 1)
          launch_lmhead<256, 64, 4, 1, 64, 1, 1>(a, L, ws, s, k, start, stop);
        else
          launch_lmhead<256, 64, 4, 1, 64, 2, 0>(a, L, ws, s, k, start, stop);
        break;
      case 128: launch_lmhead<256, 128, 2, 2, 64, 3, 3>(a, L, ws, s, k, start, stop); break;
      case 192: launch_lmhead<256, 192, 2, 2, 64, 2, 2>(a, L, ws, s, k, start, stop); break;
      default: launch_lmhead<256, 256, 2, 2, 64, 2, 2>(a, L, ws, s, k, start, stop); break;
    }
  }
  if (int rc = launch_status("k_lmhead_partial")) return rc;

  const AcceptArgs acc = accept_args(a, L, ws, conf);
  const float* rec_m = reinterpret_cast<const float*>(ws + L.off_rec_m);
  const float* rec_s = reinterpret_cast<const float*>(ws + L.off_rec_s);
  const int32_t* rec_a = reinterpret_cast<const int32_t*>(ws + L.off_rec_a);
  int32_t* cnt = reinterpret_cast<int32_t*>(ws + L.off_cnt);
  if (a->B <= kFusedMaxB) {
    k_merge_accept<<<(a->N + kFinishWaves - 1) / kFinishWaves, kFinishWaves * kWave, 0, s>>>(
        L.S, rec_m, rec_s, rec_a, a->row_max, a->row_lse, a->row_argmax, cnt, acc);
    return launch_status("k_merge_accept");
  }
  k_slab_merge<<<(a->N + kMergeRowsPerBlock - 1) / kMergeRowsPerBlock,
                 kMergeRowsPerBlock * kWave, 0, s>>>(
      a->N, L.S, rec_m, rec_s, rec_a, a->row_max, a->row_lse, a->row_argmax, a->B,
      a->req_offsets, cnt + a->B);
  if (int rc = launch_status("k_slab_merge")) return rc;
  k_tree_accept<<<a->B, kWave, 0, s>>>(cnt + a->B, acc);
  return launch_status("k_tree_accept");
}

extern "C" int asv_k1_plan(int32_t N, int32_t V, int32_t cus, int32_t tile_rows,
                           asv_k1_launch* launches, int32_t* n_launches) {
  if (N < 1 || V < 1 || cus < 1 || !grid_ok(N, V) || !launches || !n_launches)
    return ASV_EINVAL;
  Tile forced = Tile::kRows64;
  if (tile_rows != 0 && !forced_tile(tile_rows, &forced)) return ASV_EINVAL;
  const int S = (V + kSlab - 1) / kSlab;
  const K1Plan plan = tile_rows != 0 ? K1Plan{forced, forced, S} : plan_k1(N, S, cus);
  *n_launches = k1_launches(N, S, cus, plan, launches);
  return ASV_OK;
}

extern "C" int asv_verify(const asv_verify_args* a, void* workspace, uint64_t workspace_bytes,
                          void* stream) {
  return asv_verify_tuned(a, nullptr, workspace, workspace_bytes, stream);
}

extern "C" int asv_verify_noalloc(const asv_verify_args* a, void* stream) {
  if (!a || !sizes_ok(a->B, a->N, a->H, a->V)) return ASV_EINVAL;
  if (a->B == 0) return asv_verify_tuned(a, nullptr, nullptr, 0, stream);
  const size_t need = layout(a->B, a->N, a->V).bytes;
  if (need > ASV_STATIC_SCRATCH_BYTES) {
    snprintf(g_last_error, sizeof(g_last_error),
             "asv_verify_noalloc: %zu workspace bytes needed, the static scratch holds %u",
             need, ASV_STATIC_SCRATCH_BYTES);
    return ASV_ESCRATCH;
  }
  void* ws = scratch_address();
  if (!ws) return ASV_EHIP;
  return asv_verify_tuned(a, nullptr, ws, ASV_STATIC_SCRATCH_BYTES, stream);
}

extern "C" int asv_packed_lm_head_bytes(int32_t V, int32_t H, uint64_t* bytes) {
  if (!bytes || !packed_size(V, H, kPackRowsTarget, bytes)) return ASV_EINVAL;
  return ASV_OK;
}

extern "C" int asv_pack_lm_head(const uint16_t* w, int32_t V, int32_t H, uint16_t* packed,
                                uint64_t packed_bytes, void* stream) {
  return pack_tiles<kPackRowsTarget>(w, V, H, packed, packed_bytes, stream);
}

extern "C" int asv_packed_draft_head_bytes(int32_t V, int32_t H, uint64_t* bytes) {
  if (!bytes || V < kTopK || !packed_size(V, H, 128, bytes)) return ASV_EINVAL;
  return ASV_OK;
}

extern "C" int asv_pack_draft_head(const uint16_t* w, int32_t V, int32_t H, uint16_t* packed,
                                   uint64_t packed_bytes, void* stream) {
  if (V < kTopK) return ASV_EINVAL;
  return pack_tiles<kPackRowsDraft>(w, V, H, packed, packed_bytes, stream);
}

extern "C" int asv_draft_workspace_bytes(int32_t B, int32_t H, int32_t V, uint64_t* bytes) {
  if (!bytes || !draft_sizes_ok(B, H, V)) return ASV_EINVAL;
  *bytes = draft_layout(B, V).bytes;
  return ASV_OK;
}

extern "C" int asv_draft_step_tuned(const asv_draft_args* a, const asv_tuning* tuning,
                                    void* workspace, uint64_t workspace_bytes, void* stream) {
  if (!a || !draft_sizes_ok(a->B, a->H, a->V) || a->step < 0) return ASV_EINVAL;
  const asv_tuning tu = tuning ? *tuning : asv_tuning{nullptr, nullptr, 0};
  if (tu.tile_rows != 0) return ASV_EINVAL;
  if (a->w_draft_layout != ASV_W_ROW_MAJOR && a->w_draft_layout != ASV_W_PACKED)
    return ASV_EINVAL;
  uint64_t packed_bytes = 0;
  if (a->w_draft_layout == ASV_W_PACKED && !packed_size(a->V, a->H, 128, &packed_bytes))
    return ASV_EINVAL;
  if (a->B == 0) return ASV_OK;
  if (!a->hidden || !a->w_draft || !a->tree || !a->topk_id || !a->topk_logp || !a->row_lse ||
      !a->front_tok)
    return ASV_EINVAL;
  if (!aligned16(a->hidden) || !aligned16(a->w_draft)) return ASV_EINVAL;
  if (!a->state && a->step == 0) {
    const int ns = a->shape[0], tk = a->shape[1], nd = a->shape[2];
    if (!(ns >= 1 && tk >= 1 && tk <= kTopK && nd >= 1 && ns <= kPoolMax &&
          tk + (ns - 1) * tk * tk <= kPoolMax))
      return ASV_EINVAL;
  }
  const DraftLayout L = draft_layout(a->B, a->V);
  if (!workspace || workspace_bytes < L.bytes ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return ASV_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  (void)hipGetLastError();
  // timing events (measurement only): the start and the end of the draft LM head's launch
  const hipEvent_t ev_begin = reinterpret_cast<hipEvent_t>(tu.begin_event);
  const hipEvent_t ev_end = reinterpret_cast<hipEvent_t>(tu.end_event);
  switch (pick_draft_tile(a->B * kTopK)) {
    // <vocab rows, draft rows, waves along vocab, waves along rows, K per stage, ring depth>
    case DraftTile::kRows32:
      launch_draft<64, 32, 2, 1, 64, 4>(a, L, ws, s, ev_begin, ev_end);
      break;
    case DraftTile::kRows64:
      launch_draft<64, 64, 2, 2, 64, 4>(a, L, ws, s, ev_begin, ev_end);
      break;
    case DraftTile::kRows128:
      launch_draft<128, 128, 2, 4, 64, 3>(a, L, ws, s, ev_begin, ev_end);
      break;
  }
  if (int rc = launch_status("k_draft_partial")) return rc;
  DraftGrowArgs g;
  g.B = a->B;
  g.S = L.S;
  g.step = a->step;
  g.rec_k = reinterpret_cast<const uint64_t*>(ws + L.off_k);
  g.rec_s = reinterpret_cast<const float*>(ws + L.off_s);
  g.vocab_map = a->vocab_map;
  g.state = a->state;
  for (int k = 0; k < 3; ++k) g.shape[k] = a->shape[k];
  g.tree = a->tree;
  g.topk_id = a->topk_id;
  g.topk_logp = a->topk_logp;
  g.row_lse = a->row_lse;
  g.front_tok = a->front_tok;
  g.draft_conf = a->draft_conf;
  k_draft_grow<<<a->B, kDraftThreads, 0, s>>>(g);
  return launch_status("k_draft_grow");
}

extern "C" int asv_draft_step(const asv_draft_args* a, void* workspace, uint64_t workspace_bytes,
                              void* stream) {
  return asv_draft_step_tuned(a, nullptr, workspace, workspace_bytes, stream);
}

extern "C" int asv_draft_prune(const asv_draft_tree* tree, int32_t B, const int32_t* root_tok,
                               int32_t n_cap, int32_t* parent, int32_t* draft_tok,
                               int32_t* req_offsets, int32_t* req_status, void* stream) {
  if (B < 0 || n_cap < 0) return ASV_EINVAL;
  if (B == 0) return ASV_OK;
  if (!tree || !parent || !draft_tok || !req_offsets || !req_status) return ASV_EINVAL;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  k_draft_prune<<<B, kPruneThreads, 0, s>>>(tree, root_tok, n_cap, parent, draft_tok,
                                            req_offsets, req_status);
  return launch_status("k_draft_prune");
}

extern "C" int asv_tree_meta(const int32_t* parent, const int32_t* req_offsets, int32_t B,
                             int32_t N, const int32_t* pos_base, int32_t mask_words,
                             int32_t* pos, uint32_t* mask, int32_t* req_status, void* stream) {
  if (B < 0 || N < B || (B == 0) != (N == 0)) return ASV_EINVAL;
  if (B == 0) return ASV_OK;
  if (!parent || !req_offsets || !req_status || (mask && mask_words < 1)) return ASV_EINVAL;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  k_tree_meta<<<B, kMetaThreads, 0, s>>>(parent, req_offsets, B, N, pos_base, mask_words, pos,
                                         mask, req_status);
  return launch_status("k_tree_meta");
}

extern "C" int asv_commit(const asv_commit_args* a, void* stream) {
  if (!a || a->B < 0 || a->N < a->B || (a->B == 0) != (a->N == 0)) return ASV_EINVAL;
  if (a->B == 0) return ASV_OK;
  if (!a->req_offsets || !a->draft_tok || !a->accepted_len || !a->accepted_path ||
      !a->bonus_token || !a->commit_off || !a->commit_tok || !a->commit_row || !a->req_status)
    return ASV_EINVAL;
  if (a->row_src) {
    if (!a->row_dst || a->row_bytes <= 0 || a->row_bytes % 4 != 0) return ASV_EINVAL;
    if ((reinterpret_cast<uintptr_t>(a->row_src) | reinterpret_cast<uintptr_t>(a->row_dst)) & 3)
      return ASV_EINVAL;
  }
  CommitArgs c;
  c.B = a->B;
  c.N = a->N;
  c.off = a->req_offsets;
  c.tok = a->draft_tok;
  c.acc_len = a->accepted_len;
  c.path = a->accepted_path;
  c.bonus = a->bonus_token;
  c.c_off = a->commit_off;
  c.c_tok = a->commit_tok;
  c.c_row = a->commit_row;
  c.src = static_cast<const char*>(a->row_src);
  c.dst = static_cast<char*>(a->row_dst);
  c.row_bytes = a->row_bytes;
  c.status = a->req_status;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  k_commit<<<dim3(a->B, c.src ? kCommitSplit : 1), kCommitThreads, 0, s>>>(c);
  return launch_status("k_commit");
}
