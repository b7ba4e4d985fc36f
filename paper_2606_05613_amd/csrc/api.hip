// C ABI of libbkmoo: argument checks, workspace carving and stream-ordered
// launches of schedule -> Gram -> solve -> combine.  Nothing here allocates,
// frees or synchronises (except bkmoo_read_device_error, a diagnostic).
// bkmoo_resolve_noalloc runs bkmoo_resolve on a fixed-size device array of
// this file instead of a caller's workspace.
#include <atomic>
#include <mutex>

#include "bkmoo.h"
#include "internal.h"
#include "refill.h"

namespace bkmoo {

namespace {

std::atomic<int> g_grid_override{0};
std::atomic<int> g_resolve_path{0};            // 0 automatic, BKMOO_PATH_TWO_PASS, BKMOO_PATH_HYBRID
std::atomic<uint32_t> g_spin_limit{1u << 22};  // polls of the cooperative path's bounded waits

constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];

// Scratch of bkmoo_resolve_noalloc: the workspace of one resolve, up to
// kScratchBytes.  Each device holds its own copy, from when the library's
// code object is loaded there until the process ends.  Host code never uses
// the array's name as an address (on the host it is only a handle for the
// runtime): g_scratch holds each device's address of it, looked up once per
// device with that device current.
constexpr size_t kScratchBytes = (size_t)96 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
std::atomic<void *> g_scratch[kMaxDevices];

// This device's address of `scratch` (null if it cannot be had).  Two threads
// racing on a device's first call look it up twice and store the same value.
void *scratch_on_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void *p = g_scratch[dev].load();
  if (p) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
  g_scratch[dev].store(p);
  return p;
}

bool valid_dtype(int dt) { return dt == BKMOO_F32 || dt == BKMOO_BF16; }

// Shapes shared by gram / combine / resolve.
bkmoo_status check_shape(int32_t K, int64_t N, int32_t B, int dt) {
  if (K < kMinK || N < 0 || B < 1 || !valid_dtype(dt)) return BKMOO_EINVAL;
  if (K > kMaxK) return BKMOO_EUNSUPPORTED;
  return BKMOO_OK;
}

// Row pointers: non-null, naturally aligned.  128-bit loads need every row
// at the same 16-byte phase; `shift` is then the first element index whose
// address is 16-byte aligned, modulo the vector width.
bkmoo_status check_rows(int32_t K, const void *const *grads, int dt, int64_t N, int *shift,
                        bool *vec) {
  if (!grads) return BKMOO_EINVAL;
  const uintptr_t eb = (uintptr_t)elem_bytes(dt);
  const uintptr_t a0 = (uintptr_t)grads[0];
  bool same_phase = true;
  for (int i = 0; i < K; ++i) {
    const uintptr_t a = (uintptr_t)grads[i];
    if ((N > 0 && a == 0) || a % eb != 0) return BKMOO_EINVAL;
    if (a % 16 != a0 % 16) same_phase = false;
  }
  *shift = (int)(((16 - a0 % 16) % 16) / eb);
  *vec = same_phase;
  return BKMOO_OK;
}

bool overlaps(uintptr_t a, size_t na, uintptr_t b, size_t nb) { return a < b + nb && b < a + na; }

bkmoo_status check_out(int32_t K, const void *const *grads, int dt, int64_t N, const void *out,
                       int out_dt, int shift, bool *vec) {
  if (!valid_dtype(out_dt)) return BKMOO_EINVAL;
  const uintptr_t o = (uintptr_t)out;
  const uintptr_t eo = (uintptr_t)elem_bytes(out_dt);
  if ((N > 0 && o == 0) || o % eo != 0) return BKMOO_EINVAL;
  const size_t nbo = (size_t)N * eo, nbi = (size_t)N * elem_bytes(dt);
  for (int i = 0; i < K; ++i) {
    const uintptr_t r = (uintptr_t)grads[i];
    if (r == o && out_dt == dt) continue;  // exact in-place update of one row
    if (N > 0 && overlaps(o, nbo, r, nbi)) return BKMOO_EINVAL;
  }
  // vector stores: V outputs at out + (shift + m V) * s_out, 8 or 16 bytes wide
  const uintptr_t width = (uintptr_t)vec_elems(dt) * eo < 16 ? (uintptr_t)vec_elems(dt) * eo : 16;
  if ((o + (uintptr_t)shift * eo) % width != 0) *vec = false;
  return BKMOO_OK;
}

bool is_exact(int method) { return method == BKMOO_MGDA_EXACT || method == BKMOO_CAGRAD_EXACT; }

bkmoo_status check_hparams(int method, const bkmoo_hparams *hp) {
  if (method < BKMOO_MGDA || method > BKMOO_CAGRAD_EXACT) return BKMOO_EINVAL;
  if (method == BKMOO_MEAN || method == BKMOO_MGDA_EXACT) return BKMOO_OK;
  if (!hp) return BKMOO_EINVAL;
  if ((method == BKMOO_MGDA || method == BKMOO_CAGRAD) && (hp->max_iter < 0 || hp->max_iter > 1000000))
    return BKMOO_EINVAL;
  if ((method == BKMOO_CAGRAD || method == BKMOO_CAGRAD_EXACT) &&
      !(hp->cagrad_c >= 0.0 && hp->cagrad_c < 1.0))
    return BKMOO_EINVAL;
  return BKMOO_OK;
}

// K beyond what the method supports (exact solvers enumerate 2^K - 1 supports).
bool k_unsupported(int K, int method) { return K > kMaxK || (is_exact(method) && K > kExactMaxK); }

bkmoo_status hip_status(hipError_t e) { return e == hipSuccess ? BKMOO_OK : BKMOO_EHIP; }

struct Carved {
  uint32_t *err;
  int64_t *chunk_start;
  double *gram;
  float *weights;
  double *partials;
  int64_t *group_start;
  double *groups;
  uint32_t *sync;
};

Carved carve(void *ws, const Layout &L) {
  char *base = static_cast<char *>(ws);
  return Carved{reinterpret_cast<uint32_t *>(base + L.err),
                reinterpret_cast<int64_t *>(base + L.chunk_start),
                reinterpret_cast<double *>(base + L.gram), reinterpret_cast<float *>(base + L.weights),
                reinterpret_cast<double *>(base + L.partials),
                reinterpret_cast<int64_t *>(base + L.group_start),
                reinterpret_cast<double *>(base + L.groups), reinterpret_cast<uint32_t *>(base + L.sync)};
}

// The cooperative kernel's grid (Grid: hybrid_grid) on the current device,
// computed once per device and instantiation; 0 if the kernel cannot run
// there.
template <int (*Grid)(int, int, int)>
int cached_grid(int K, int dt, int out_dt) {
  static std::atomic<int> cache[kMaxDevices][kMaxK - 1][2][2];  // K-2, dt, out_dt: 0 unknown, -1 none
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    const int g = Grid(K, dt, out_dt);
    return g > 0 ? g : 0;
  }
  std::atomic<int> &c = cache[dev][K - 2][dt][out_dt];
  int g = c.load();
  if (g == 0) {
    g = Grid(K, dt, out_dt);
    c.store(g > 0 ? g : -1);
  }
  return g > 0 ? g : 0;
}

// The pipelined, partly resident path pays when each bucket carries enough
// data to amortise its hand-off (reduction, solve, weights) and a fair
// share of each segment stays on chip.  A bucket's solve runs on one
// wavefront while the data workgroups stream the next bucket; its estimated
// latency L (solve_latency_us) raises the bucket size needed:
//   all K rows of the average bucket >= 24 MiB + 4 MiB per us of L,
// at least 8 buckets, at least 10% of a bucket kept on chip.  Every
// crossover measured on MI355X (K = 2..4 bf16, buckets of 4-400 MiB per
// row, mean, PCGrad, MGDA and CAGrad with 20 or 100 iterations) falls on
// the side this predicts or is a near-tie, except some K = 2 wins left to
// the two passes (the K = 2 solves run faster than L assumes): for the mean
// method the
// two passes win at 16-20 MiB (all rows) and lose from 28 MiB (K=4: 5%
// slower at 24 MiB, 12% faster at 28); MGDA FW-20 at K=4 (L = 5.6 us)
// loses at 32 MiB, ties at 48 and wins 11-21% from 64; CAGrad FW-20 (L =
// 17.6 us) loses at 64 MiB and wins at 100; MGDA FW-100 (L = 28 us) ties at
// 100 MiB and wins at 200; buckets above ~150 MiB per row keep less than 10%
// on chip and lose.
constexpr int kHybridMinBuckets = 8;
constexpr double kHybridBaseMiB = 24.0;   // all K rows, no solve
constexpr double kHybridBaseMiBPerRow = 6.0;  // ... and at least this per row (K > 4)
constexpr double kHybridMiBPerUs = 4.0;   // per microsecond of solve latency
constexpr double kHybridMinHeld = 0.1;    // fraction of a bucket kept on chip

// Estimated latency of one bucket's solve on one wavefront (microseconds):
// 0.28 us per Frank-Wolfe iteration for MGDA and 0.9 us per dual iteration
// for CAGrad measured at K = 4, chains growing with K; PCGrad's K(K-1)
// projections are short.
double solve_latency_us(int method, int K, int iters) {
  if (method == BKMOO_MGDA) return 0.07 * K * iters;
  if (method == BKMOO_CAGRAD) return 0.22 * K * iters;
  if (method == BKMOO_PCGRAD) return 0.1 * K * K;
  return 0.0;
}

// How the hybrid kernel lays out a bucket for a call with a solve.  Two
// workgroups share each CU; the one dispatched second loses the wave
// arbiter and arrives last at every bucket, and the four data workgroups
// that share a CU with a solver lose it to the solve (which runs at raised
// priority).  Two remedies: a segment skew (the first-dispatched data
// workgroups take 35% more) and leaving the solvers' CU mates without a
// segment.  Measured on MI355X, 25 MiB buckets per row (613), bf16, ms per
// call, skew / mates empty / neither:
//   K=4 MGDA FW-15 17.33 / 18.03 / 17.89, FW-20 17.45 / 17.98 / 18.36,
//       FW-40 19.04 / 18.51 / 20.78, FW-100 25.40 / 24.55 / 27.48,
//       CAGrad FW-5 17.51 / 17.78 / 17.92, FW-10 17.77 / 17.76 / 18.75,
//       FW-20 19.75 / 19.10 / 20.82, MGDA FW-10 17.91 / 17.64 / 17.70
//   K=5 MGDA FW-20 27.15 / 25.96 / 25.76, CAGrad FW-20 27.58 / 24.24 / 25.62
//   K=6 MGDA FW-20 26.39 / 25.14 / 25.99, CAGrad FW-20 28.24 / 27.01 / 29.31
//   K=7 MGDA FW-20 31.56 / 30.59 / 31.34, CAGrad FW-20 33.77 / 32.88 / 35.81
//   K=8 MGDA FW-20 37.96 / 35.83 / 36.06, CAGrad FW-20 38.95 / 37.73 / 40.49
//   K=3 CAGrad FW-20 (no skew below K=4) 15.10 mates empty / 16.66 neither
// and no difference for the mean method, PCGrad or solves under ~3 us.  So
// the skew is for K = 4 solves of 4-9 us, and the mates go without data for
// every other solve of 3 us or more.  The skew also needs rows of at most
// 32 MiB per bucket (at 50 MiB it slowed CAGrad by 5%) and second
// workgroups whose shares still fill what they keep on chip.
constexpr int kHybridSkewPm = 350;
constexpr double kHybridSkewMaxRowBytes = 32.0 * (1 << 20);
constexpr double kHybridSkewMinUs = 4.0, kHybridSkewMaxUs = 9.0;
constexpr double kHybridLightMinUs = 3.0;

int hybrid_skew_pm(int K, int dt, int out_dt, int method, int iters, int64_t N, int B, int grid) {
  if (K != 4 || (method != BKMOO_MGDA && method != BKMOO_CAGRAD) || iters <= 0 || B <= 0) return 0;
  const double lat = solve_latency_us(method, K, iters);
  if (lat < kHybridSkewMinUs || lat >= kHybridSkewMaxUs) return 0;
  const double avg = (double)N / B;
  if (avg * elem_bytes(dt) > kHybridSkewMaxRowBytes) return 0;
  const int gd = hybrid_data_workgroups(grid), older = hybrid_older_workgroups(grid);
  if (older <= 0 || older >= gd) return 0;
  // the second workgroups' segments must still fill their on-chip share
  const int64_t unit = hybrid_unit_elems(dt), nb = hybrid_held_elems(K, dt, out_dt) / unit;
  const int64_t nu = (int64_t)(avg / unit);
  const int64_t co = (nu * (1000 + kHybridSkewPm) + (int64_t)gd * 1000 - 1) / ((int64_t)gd * 1000);
  const int64_t rest = nu - (int64_t)older * co;
  const int64_t cy = rest > 0 ? (rest + (gd - older) - 1) / (gd - older) : 0;
  return cy >= nb ? kHybridSkewPm : 0;
}

// The hybrid kernel's layout for one call (grid from hybrid_grid).
HybLayout hybrid_layout(int K, int dt, int out_dt, int method, int iters, int64_t N, int B, int grid) {
  HybLayout L{hybrid_data_workgroups(grid), hybrid_older_workgroups(grid), 0, 0};
  if (L.older <= 0 || L.older + kHybridSolvers >= L.nslots) return L;
  L.skew_pm = hybrid_skew_pm(K, dt, out_dt, method, iters, N, B, grid);
  if (L.skew_pm == 0 && (method == BKMOO_MGDA || method == BKMOO_CAGRAD) &&
      solve_latency_us(method, K, iters) >= kHybridLightMinUs) {
    L.light = 1;
    L.nslots -= kHybridSolvers;
  }
  return L;
}

// Workgroups for the pipelined, partly resident path, or 0 when it should
// not be used.  Its partial Grams need two slots per data workgroup, and a
// segment (about N / data workgroups elements at most) must stay within one
// 32-bit buffer range.
int choose_hybrid(int K, int dt, int out_dt, int64_t N, int B, bool vec, int method, int iters,
                  int64_t cap_slots) {
  const int mode = g_resolve_path.load();
  if (mode == BKMOO_PATH_TWO_PASS || mode == BKMOO_PATH_REFILL || K > kHybridMaxK || !vec || is_exact(method))
    return 0;
  const int g = cached_grid<hybrid_grid>(K, dt, out_dt);
  if (g <= 0) return 0;
  const int gd = hybrid_data_workgroups(g);
  if (2 * (int64_t)gd > cap_slots) return 0;
  if ((N / gd + 2 * 4096) * (int64_t)elem_bytes(dt) >= ((int64_t)1 << 31)) return 0;
  if (mode == BKMOO_PATH_HYBRID) return g;
  const double avg_elems = (double)N / B;
  const double bucket_bytes = avg_elems * K * elem_bytes(dt);
  const double held = (double)hybrid_held_elems(K, dt, out_dt) * gd / (avg_elems > 1.0 ? avg_elems : 1.0);
  const double base_mib = kHybridBaseMiB > kHybridBaseMiBPerRow * K ? kHybridBaseMiB : kHybridBaseMiBPerRow * K;
  const double min_bytes = (base_mib + kHybridMiBPerUs * solve_latency_us(method, K, iters)) * (1 << 20);
  return B >= kHybridMinBuckets && bucket_bytes >= min_bytes && held >= kHybridMinHeld ? g : 0;
}

// Groups of data workgroups for the single-buffer path: group g takes
// buckets g, g + groups, ..., so a bucket's hand-off hides behind a round of
// `groups` buckets of streaming instead of one.  A round of about
// kRefillRoundMiB (all rows) is long enough to hide it and short enough
// for the streamed part to be re-read from the 256 MB Infinity Cache;
// beyond ~kRefillMaxRoundMiB the re-reads miss.  Measured on MI355X (ms per
// call, two passes / refill at the groups the rule picks; best nearby
// count in brackets): K=10 fp32 1.72B elements, 1 MiB per row CAGrad FW-20
// 25.3 / 18.6 (G=18; 14: 18.6, 22: 22.5, 8: 33.6), MGDA 25.1 / 18.5,
// PCGrad 25.1 / 18.3; 5 MiB CAGrad 23.2 / 18.1 (G=4; 3: 19.9, 5: 20.1),
// MGDA 22.7 / 18.2, PCGrad 22.7 / 17.9; 25 MiB CAGrad 25.1 / 22.3 (G=1;
// 2: 25.7); 100 MiB (G=1, a 1 GB round) 25.1 / 24.7.  K=4 bf16 2.1B
// elements, 1 MiB MGDA 6.6 / 4.5 (G=32), CAGrad 6.7 / 5.1; 5 MiB MGDA
// 6.6 / 4.5 (G=9; 6: 4.3), CAGrad 6.6 / 4.7.  K=8 bf16 1.07B elements,
// 1 MiB MGDA 6.3 / 4.9 (G=24), CAGrad 6.3 / 5.0; 5 MiB MGDA 6.3 / 4.9
// (G=4), CAGrad 6.3 / 5.3.  With one group (a bucket of more than ~120
// MiB) the cap does not apply: the re-read part of a bucket misses as it
// does on the two passes, and the kept part still saves its second read.
// Two passes / refill, MGDA FW-20: K=4 bf16 100 MiB per row 6.57 / 5.75,
// K=4 fp32 400 MiB 3.32 / 3.21, K=2 bf16 400 MiB 3.70 / 3.59, K=6 bf16
// 100 MiB 4.78 / 4.65, K=8 bf16 100 MiB 6.32 / 6.26, K=9 fp32 100 MiB
// 3.92 / 3.40, K=10 bf16 100 MiB 8.54 / 8.04 (CAGrad and the mean alike).
constexpr double kRefillRoundMiB = 180.0;
constexpr double kRefillMaxRoundMiB = 300.0;
// A round must also cover the hand-off: at least this much, plus this much
// per microsecond of estimated solve latency.
constexpr double kRefillMinRoundMiB = 64.0, kRefillMiBPerUs = 2.0;
// Where both cooperative kernels can run (K <= 8, large buckets) the
// two-buffer one is as fast or faster at K > 4 and for short solves; at
// K <= 4 a solve of a few microseconds shows in its hand-off, while the
// refill kernel's groups hide it.  Measured on MI355X, bf16, ms, two-buffer
// / refill at the rule's G: K=4 25 MiB per row (613 buckets) MGDA FW-20
// 17.36 / 16.82 (G=2), CAGrad FW-20 19.02 / 16.70, mean 16.06 / 17.02,
// PCGrad 16.09 / 17.06; K=4 50 MiB (82) MGDA 5.34 / 4.98 (G=1), CAGrad
// 5.24 / 5.02; K=4 12.5 MiB (328) MGDA 5.66 / 4.52 (G=4); K=3 25 MiB (328)
// MGDA 5.24 / 4.79 (G=2), CAGrad 5.48 / 5.04; K=2 25 MiB (328) MGDA FW-20
// (2.8 us) 5.52 / 5.83 (G=4), CAGrad 6.83 / 5.70; K=6 MGDA 3.42 / 3.75; K=8
// CAGrad FW-20 36.4 / 39.4 (G=1), 41.0 (G=2).  With nine kept register
// vectors at K=4 (one process each, ms): K=4 25 MiB mean 16.03 / 17.09,
// PCGrad 16.15 / 16.91, MGDA FW-20 17.39 / 16.58, CAGrad 18.97 / 16.94;
// K=4 fp32 GPT-2 shape (19 buckets) PCGrad 0.54 / 0.56, CAGrad 0.63 /
// 0.59; K=2 25 MiB mean 5.59 / 5.86, MGDA 5.47 / 5.83, CAGrad 6.79 / 5.70;
// K=3 25 MiB mean 5.21 / 5.01, PCGrad 5.26 / 4.93, MGDA 5.23 / 4.78,
// CAGrad 5.49 / 5.04: at K = 3 the refill kernel wins for every method.
constexpr double kRefillOverHybridUs = 4.0;

int refill_groups(int K, int dt, int64_t N, int B) {
  const double bucket_mib = (double)N / B * K * elem_bytes(dt) / (1 << 20);
  int g = (int)(kRefillRoundMiB / (bucket_mib > 1e-9 ? bucket_mib : 1e-9) + 0.5);
  g = g < 1 ? 1 : g > kRefMaxGroups ? kRefMaxGroups : g;
  return g < B ? g : (B > 0 ? B : 1);
}

// Workgroups for the single-buffer pipelined path if it can run and, unless
// forced, its own size rule holds (the choice against the two-buffer path
// is made in pick_path); else 0.
int choose_refill(int K, int dt, int out_dt, int64_t N, int B, bool vec, int method, int iters) {
  const int mode = g_resolve_path.load();
  if (mode == BKMOO_PATH_TWO_PASS || mode == BKMOO_PATH_HYBRID || K > kRefillMaxK || !vec || is_exact(method))
    return 0;
  const int g = cached_grid<refill_grid>(K, dt, out_dt);
  if (g <= 0) return 0;
  const int groups = refill_groups(K, dt, N, B);
  // a segment (at most N over one group's data workgroups) within one
  // 32-bit buffer range
  if ((N / ((g - refill_solvers(groups)) / groups) + 2 * 4096) * (int64_t)elem_bytes(dt) >= ((int64_t)1 << 31))
    return 0;
  if (mode == BKMOO_PATH_REFILL) return g;
  if (B < kHybridMinBuckets) return 0;
  const double round_mib = (double)N / B * K * elem_bytes(dt) / (1 << 20) * groups;
  const double min_mib = kRefillMinRoundMiB + kRefillMiBPerUs * solve_latency_us(method, K, iters);
  return round_mib >= min_mib && (round_mib <= kRefillMaxRoundMiB || groups == 1) ? g : 0;
}

// The path bkmoo_resolve takes and its grid (0 for the two passes).
int pick_path(int K, int dt, int out_dt, int64_t N, int B, bool vec, int method, int iters, int64_t cap_slots,
              int *grid) {
  const int rg = choose_refill(K, dt, out_dt, N, B, vec, method, iters);
  const int hg = choose_hybrid(K, dt, out_dt, N, B, vec, method, iters, cap_slots);
  const bool prefer_refill = K == 3 || (K <= 4 && solve_latency_us(method, K, iters) >= kRefillOverHybridUs);
  if (rg > 0 && (hg <= 0 || prefer_refill || g_resolve_path.load() == BKMOO_PATH_REFILL)) {
    *grid = rg;
    return BKMOO_PATH_REFILL;
  }
  if (hg > 0) {
    *grid = hg;
    return BKMOO_PATH_HYBRID;
  }
  *grid = 0;
  return BKMOO_PATH_TWO_PASS;
}

// bkmoo_resolve's argument checks (everything but the workspace); the
// 16-byte row phase and whether rows and output allow vector accesses.
bkmoo_status check_resolve(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                           const int64_t *bucket_offsets, bkmoo_method method, const bkmoo_hparams *hp,
                           const void *out, bkmoo_dtype out_dt, int *shift, bool *vec_in, bool *vec_out) {
  bkmoo_status st = check_shape(K, N, B, dt);
  if (st != BKMOO_OK) return st;
  if ((st = check_rows(K, grads, dt, N, shift, vec_in)) != BKMOO_OK) return st;
  *vec_out = *vec_in;
  if ((st = check_out(K, grads, dt, N, out, out_dt, *shift, vec_out)) != BKMOO_OK) return st;
  if ((st = check_hparams(method, hp)) != BKMOO_OK) return st;
  if (k_unsupported(K, method)) return BKMOO_EUNSUPPORTED;
  return bucket_offsets ? BKMOO_OK : BKMOO_EINVAL;
}

// bkmoo_resolve's work, on the workspace given (see bkmoo_resolve).
bkmoo_status resolve_impl(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                          const int64_t *bucket_offsets, bkmoo_method method, const bkmoo_hparams *hp,
                          void *out, bkmoo_dtype out_dt, double *gram, float *weights, double *aux,
                          void *workspace, size_t ws_bytes, hipStream_t stream);

}  // namespace

int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 1;
  if (dev < kMaxDevices) {
    const int cached = g_cu_count[dev].load(std::memory_order_relaxed);
    if (cached > 0) return cached;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
    n = 1;
  if (dev < kMaxDevices) g_cu_count[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace bkmoo

using namespace bkmoo;

extern "C" {

bkmoo_status bkmoo_workspace_size(int32_t K, int64_t N, int32_t B, bkmoo_dtype dt, size_t *bytes) {
  if (!bytes) return BKMOO_EINVAL;
  const bkmoo_status st = check_shape(K, N, B, dt);
  if (st != BKMOO_OK) return st;
  *bytes = layout(K, N, B, dt).total;
  return BKMOO_OK;
}

bkmoo_status bkmoo_gram(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                        const int64_t *bucket_offsets, double *gram, void *workspace,
                        size_t ws_bytes, hipStream_t stream) {
  bkmoo_status st = check_shape(K, N, B, dt);
  if (st != BKMOO_OK) return st;
  int shift = 0;
  bool vec = false;
  if ((st = check_rows(K, grads, dt, N, &shift, &vec)) != BKMOO_OK) return st;
  if (!bucket_offsets || !gram || !workspace) return BKMOO_EINVAL;
  const Layout L = layout(K, N, B, dt);
  if (ws_bytes < L.total) return BKMOO_EWORKSPACE;
  const Carved w = carve(workspace, L);
  hipError_t e = launch_schedule(bucket_offsets, B, N, gram_chunk_elems(K, dt), w.chunk_start,
                                 w.group_start, w.err, nullptr, 0, stream);
  if (e != hipSuccess) return BKMOO_EHIP;
  const StreamArgs a{K, (int)dt, grads, N, B, bucket_offsets, w.chunk_start, w.group_start, w.err,
                     shift, vec, g_grid_override.load()};
  return hip_status(launch_gram(a, w.partials, w.groups, L.cap_groups, gram, stream));
}

bkmoo_status bkmoo_solve(int32_t K, int32_t B, const double *gram, bkmoo_method method,
                         const bkmoo_hparams *hp, float *weights, double *aux, hipStream_t stream) {
  if (K < kMinK || B < 1) return BKMOO_EINVAL;
  if (K > kMaxK) return BKMOO_EUNSUPPORTED;
  if (!gram || !weights) return BKMOO_EINVAL;
  const bkmoo_status st = check_hparams(method, hp);
  if (st != BKMOO_OK) return st;
  if (k_unsupported(K, method)) return BKMOO_EUNSUPPORTED;
  const int iters = hp ? hp->max_iter : 0;
  const double c = hp ? hp->cagrad_c : 0.0;
  const int8_t *order = hp ? hp->pcgrad_order : nullptr;
  return hip_status(launch_solve(K, B, gram, (int)method, iters, c, order, weights, aux, stream));
}

bkmoo_status bkmoo_combine(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                           const int64_t *bucket_offsets, const float *weights, void *out,
                           bkmoo_dtype out_dt, void *workspace, size_t ws_bytes, hipStream_t stream) {
  bkmoo_status st = check_shape(K, N, B, dt);
  if (st != BKMOO_OK) return st;
  int shift = 0;
  bool vec = false;
  if ((st = check_rows(K, grads, dt, N, &shift, &vec)) != BKMOO_OK) return st;
  if ((st = check_out(K, grads, dt, N, out, out_dt, shift, &vec)) != BKMOO_OK) return st;
  if (!bucket_offsets || !weights || !workspace) return BKMOO_EINVAL;
  const Layout L = layout(K, N, B, dt);
  if (ws_bytes < L.total) return BKMOO_EWORKSPACE;
  const Carved w = carve(workspace, L);
  hipError_t e = launch_schedule(bucket_offsets, B, N, combine_chunk_elems(K, dt), w.chunk_start,
                                 nullptr, w.err, nullptr, 0, stream);
  if (e != hipSuccess) return BKMOO_EHIP;
  const StreamArgs a{K, (int)dt, grads, N, B, bucket_offsets, w.chunk_start, nullptr, w.err, shift,
                     vec, g_grid_override.load()};
  return hip_status(launch_combine(a, weights, out, (int)out_dt, stream));
}

bkmoo_status bkmoo_resolve(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                           const int64_t *bucket_offsets, bkmoo_method method,
                           const bkmoo_hparams *hp, void *out, bkmoo_dtype out_dt, double *gram,
                           float *weights, double *aux, void *workspace, size_t ws_bytes,
                           hipStream_t stream) {
  return resolve_impl(K, grads, dt, N, B, bucket_offsets, method, hp, out, out_dt, gram, weights, aux,
                      workspace, ws_bytes, stream);
}

bkmoo_status bkmoo_resolve_noalloc(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N,
                                   int32_t B, const int64_t *bucket_offsets, bkmoo_method method,
                                   const bkmoo_hparams *hp, void *out, bkmoo_dtype out_dt, double *gram,
                                   float *weights, double *aux, hipStream_t stream) {
  int shift = 0;
  bool vec_in = false, vec_out = false;
  const bkmoo_status st = check_resolve(K, grads, dt, N, B, bucket_offsets, method, hp, out, out_dt, &shift,
                                        &vec_in, &vec_out);
  if (st != BKMOO_OK) return st;
  if (layout(K, N, B, dt).total > kScratchBytes) return BKMOO_EWORKSPACE;
  void *ws = scratch_on_current_device();
  if (!ws) return BKMOO_EHIP;
  return resolve_impl(K, grads, dt, N, B, bucket_offsets, method, hp, out, out_dt, gram, weights, aux, ws,
                      kScratchBytes, stream);
}

}  // extern "C"

namespace bkmoo {
namespace {

bkmoo_status resolve_impl(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                          const int64_t *bucket_offsets, bkmoo_method method, const bkmoo_hparams *hp,
                          void *out, bkmoo_dtype out_dt, double *gram, float *weights, double *aux,
                          void *workspace, size_t ws_bytes, hipStream_t stream) {
  int shift = 0;
  bool vec_in = false, vec_out = false;
  const bkmoo_status st = check_resolve(K, grads, dt, N, B, bucket_offsets, method, hp, out, out_dt, &shift,
                                        &vec_in, &vec_out);
  if (st != BKMOO_OK) return st;
  if (!workspace) return BKMOO_EINVAL;
  const Layout L = layout(K, N, B, dt);
  if (ws_bytes < L.total) return BKMOO_EWORKSPACE;
  const Carved w = carve(workspace, L);
  double *G = gram ? gram : w.gram;
  float *W = weights ? weights : w.weights;
  const int iters = hp ? hp->max_iter : 0;
  const double c = hp ? hp->cagrad_c : 0.0;
  const int8_t *order = hp ? hp->pcgrad_order : nullptr;

  int pgrid = 0;
  const int path = pick_path(K, (int)dt, (int)out_dt, N, B, vec_in && vec_out, (int)method, iters, L.cap_chunks,
                             &pgrid);
  if (path == BKMOO_PATH_REFILL) {
    hipError_t e = launch_schedule(bucket_offsets, B, N, gram_chunk_elems(K, dt), w.chunk_start, nullptr,
                                   w.err, nullptr, 0, stream);
    if (e != hipSuccess) return BKMOO_EHIP;
    e = launch_refill(K, (int)dt, (int)out_dt, grads, bucket_offsets, B, shift, (int)method, iters, c, order,
                      G, W, aux, out, w.partials, w.sync, w.sync + B * kSyncStride, w.err, g_spin_limit.load(),
                      pgrid, refill_groups(K, (int)dt, N, B),
                      refill_temporal_slots(K, (int)dt, pgrid, refill_groups(K, (int)dt, N, B)), stream);
    return hip_status(e);
  }
  if (path == BKMOO_PATH_HYBRID) {
    const int hgrid = pgrid;
    hipError_t e = launch_schedule(bucket_offsets, B, N, gram_chunk_elems(K, dt), w.chunk_start,
                                   nullptr, w.err, w.sync, (1 + kFlagCopies) * (int64_t)B * kSyncStride, stream);
    if (e != hipSuccess) return BKMOO_EHIP;
    e = launch_hybrid(K, (int)dt, (int)out_dt, grads, bucket_offsets, B, shift, (int)method, iters, c,
                      order, G, W, aux, out, w.partials, w.sync, w.sync + B * kSyncStride, w.err, g_spin_limit.load(),
                      hgrid, hybrid_layout(K, (int)dt, (int)out_dt, (int)method, iters, N, B, hgrid), stream);
    return hip_status(e);
  }

  hipError_t e = launch_schedule(bucket_offsets, B, N, gram_chunk_elems(K, dt), w.chunk_start,
                                 w.group_start, w.err, nullptr, 0, stream);
  if (e != hipSuccess) return BKMOO_EHIP;
  StreamArgs a{K, (int)dt, grads, N, B, bucket_offsets, w.chunk_start, w.group_start, w.err, shift,
               vec_in, g_grid_override.load()};
  if ((e = launch_gram(a, w.partials, w.groups, L.cap_groups, G, stream)) != hipSuccess)
    return BKMOO_EHIP;
  if ((e = launch_solve(K, B, G, (int)method, iters, c, order, W, aux, stream)) != hipSuccess)
    return BKMOO_EHIP;
  // the combine pass cuts its own chunks (the schedule keeps the error word
  // the Gram pass's schedule set: offsets are the same)
  e = launch_schedule(bucket_offsets, B, N, combine_chunk_elems(K, dt), w.chunk_start, nullptr, w.err,
                      nullptr, 0, stream);
  if (e != hipSuccess) return BKMOO_EHIP;
  a.vec = vec_out;
  return hip_status(launch_combine(a, W, out, (int)out_dt, stream));
}

}  // namespace
}  // namespace bkmoo

extern "C" {

bkmoo_status bkmoo_slice_offsets(int32_t B, int32_t T, const int64_t *bucket_offsets,
                                 int64_t *slice_offsets, hipStream_t stream) {
  if (B < 1 || T < 1 || (int64_t)B * T > INT32_MAX) return BKMOO_EINVAL;
  if (!bucket_offsets || !slice_offsets) return BKMOO_EINVAL;
  return hip_status(launch_slice_offsets(bucket_offsets, B, T, slice_offsets, stream));
}

bkmoo_status bkmoo_gram_reduce(int32_t K, int32_t B, int32_t T, const double *partial,
                               bkmoo_slice_layout layout, double *gram, hipStream_t stream) {
  if (K < kMinK || B < 1 || T < 1) return BKMOO_EINVAL;
  if (K > kMaxK) return BKMOO_EUNSUPPORTED;
  if (!partial || !gram) return BKMOO_EINVAL;
  if (layout != BKMOO_SLICES_RANK_MAJOR && layout != BKMOO_SLICES_BUCKET_MAJOR) return BKMOO_EINVAL;
  const size_t in_bytes = sizeof(double) * (size_t)T * B * K * K;
  const size_t out_bytes = sizeof(double) * (size_t)B * K * K;
  const char *pi = reinterpret_cast<const char *>(partial), *po = reinterpret_cast<const char *>(gram);
  if (po < pi + in_bytes && pi < po + out_bytes) return BKMOO_EINVAL;
  return hip_status(launch_gram_reduce(K, B, T, partial, layout == BKMOO_SLICES_BUCKET_MAJOR ? 1 : 0,
                                       gram, stream));
}

bkmoo_status bkmoo_conflicts(int32_t K, int32_t B, const double *gram, double *cosines,
                             double *summary, int32_t *pairs, hipStream_t stream) {
  if (K < kMinK || B < 1) return BKMOO_EINVAL;
  if (K > kMaxK) return BKMOO_EUNSUPPORTED;
  if (!gram || (!cosines && !summary && !pairs)) return BKMOO_EINVAL;
  return hip_status(launch_conflicts(K, B, gram, cosines, summary, pairs, stream));
}

bkmoo_status bkmoo_resolve_traffic(int32_t K, int64_t N, int32_t B, const int64_t *offsets_host,
                                   bkmoo_dtype dt, bkmoo_dtype out_dt, bkmoo_method method, int32_t max_iter,
                                   int32_t path, uint64_t *bytes) {
  bkmoo_status st = check_shape(K, N, B, dt);
  if (st != BKMOO_OK) return st;
  if (!offsets_host || !bytes || !valid_dtype(out_dt)) return BKMOO_EINVAL;
  if (method < BKMOO_MGDA || method > BKMOO_CAGRAD_EXACT || max_iter < 0) return BKMOO_EINVAL;
  if (offsets_host[0] != 0 || offsets_host[B] != N) return BKMOO_EINVAL;
  for (int b = 0; b < B; ++b)
    if (offsets_host[b + 1] < offsets_host[b]) return BKMOO_EINVAL;
  const uint64_t s = (uint64_t)elem_bytes(dt), so = (uint64_t)elem_bytes(out_dt);
  const uint64_t once = (uint64_t)K * s * (uint64_t)N + so * (uint64_t)N;
  if (path == BKMOO_PATH_TWO_PASS) {
    *bytes = once + (uint64_t)K * s * (uint64_t)N;
    return BKMOO_OK;
  }
  if (path == BKMOO_PATH_REFILL) {
    if (K > 10) return BKMOO_EUNSUPPORTED;
    const int g = refill_grid(K, (int)dt, (int)out_dt);
    if (g <= 0) return BKMOO_EUNSUPPORTED;
    const int groups = refill_groups(K, (int)dt, N, B);
    const HybLayout lay{(g - refill_solvers(groups)) / groups, 0, 0, 0};
    const int64_t unit = hybrid_unit_elems((int)dt), held_max = refill_held_elems(K, (int)dt, (int)out_dt);
    const int64_t smin = (int64_t)refill_stream_min() * unit;
    uint64_t reread = 0;
    for (int b = 0; b < B; ++b) {  // each segment re-reads what it did not keep
      const int64_t n = offsets_host[b + 1] - offsets_host[b];
      int64_t lo, hi, nseg, ns;
      lay.segment(n, 0, unit, lo, hi, nseg);
      for (int w = 0; w < nseg; ++w) {
        lay.segment(n, w, unit, lo, hi, ns);
        const int64_t len = hi - lo, slots = (len + unit - 1) / unit;
        int64_t keep = slots * unit - smin;
        keep = keep < 0 ? 0 : keep > held_max ? held_max : keep;
        if (len > keep) reread += (uint64_t)(len - keep);
      }
    }
    *bytes = once + (uint64_t)K * s * reread;
    return BKMOO_OK;
  }
  if (path != BKMOO_PATH_HYBRID) return BKMOO_EINVAL;
  if (K > kHybridMaxK) return BKMOO_EUNSUPPORTED;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return BKMOO_EHIP;
  uint64_t reread = 0;  // elements read a second time
  {
    const int g = hybrid_grid(K, (int)dt, (int)out_dt);
    if (g <= 0) return BKMOO_EUNSUPPORTED;
    const HybLayout lay = hybrid_layout(K, (int)dt, (int)out_dt, (int)method, max_iter, N, B, g);
    const int64_t unit = hybrid_unit_elems((int)dt), held = hybrid_held_elems(K, (int)dt, (int)out_dt);
    for (int b = 0; b < B; ++b) {  // each segment re-reads what it did not keep
      const int64_t n = offsets_host[b + 1] - offsets_host[b];
      int64_t lo, hi, nseg, ns;
      lay.segment(n, 0, unit, lo, hi, nseg);
      for (int w = 0; w < nseg; ++w) {
        lay.segment(n, w, unit, lo, hi, ns);
        if (hi - lo > held) reread += (uint64_t)(hi - lo - held);
      }
    }
  }
  *bytes = once + (uint64_t)K * s * reread;
  return BKMOO_OK;
}

bkmoo_status bkmoo_read_device_error(const void *workspace, uint32_t *err, hipStream_t stream) {
  if (!workspace || !err) return BKMOO_EINVAL;
  uint32_t v = 0;
  if (hipMemcpyAsync(&v, workspace, sizeof(v), hipMemcpyDeviceToHost, stream) != hipSuccess)
    return BKMOO_EHIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return BKMOO_EHIP;
  *err = v;
  return BKMOO_OK;
}

bkmoo_status bkmoo_set_grid_override(int32_t workgroups) {
  if (workgroups < 0) return BKMOO_EINVAL;
  g_grid_override.store(workgroups);
  return BKMOO_OK;
}

bkmoo_status bkmoo_resolve_path(int32_t K, int64_t N, int32_t B, bkmoo_dtype dt, bkmoo_dtype out_dt,
                                int32_t aligned, bkmoo_method method, int32_t max_iter,
                                int32_t *path) {
  if (!path) return BKMOO_EINVAL;
  const bkmoo_status st = check_shape(K, N, B, dt);
  if (st != BKMOO_OK) return st;
  if (!valid_dtype(out_dt) || method < BKMOO_MGDA || method > BKMOO_CAGRAD_EXACT) return BKMOO_EINVAL;
  if (k_unsupported(K, method)) return BKMOO_EUNSUPPORTED;
  int grid = 0;
  *path = pick_path(K, (int)dt, (int)out_dt, N, B, aligned != 0, (int)method, max_iter,
                    layout(K, N, B, dt).cap_chunks, &grid);
  return BKMOO_OK;
}

bkmoo_status bkmoo_set_resolve_path(int32_t path) {
  if (path != 0 && path != BKMOO_PATH_TWO_PASS && path != BKMOO_PATH_HYBRID && path != BKMOO_PATH_REFILL)
    return BKMOO_EINVAL;
  g_resolve_path.store(path);
  return BKMOO_OK;
}

bkmoo_status bkmoo_set_wait_limit(uint32_t polls) {
  if (polls == 0) return BKMOO_EINVAL;
  g_spin_limit.store(polls);
  return BKMOO_OK;
}

const char *bkmoo_status_string(bkmoo_status st) {
  switch (st) {
    case BKMOO_OK: return "BKMOO_OK";
    case BKMOO_EINVAL: return "BKMOO_EINVAL: invalid argument";
    case BKMOO_EUNSUPPORTED: return "BKMOO_EUNSUPPORTED: unsupported configuration";
    case BKMOO_EWORKSPACE: return "BKMOO_EWORKSPACE: workspace too small";
    case BKMOO_EHIP: return "BKMOO_EHIP: HIP launch or runtime failure";
    default: return "BKMOO: unknown status";
  }
}

}  // extern "C"
