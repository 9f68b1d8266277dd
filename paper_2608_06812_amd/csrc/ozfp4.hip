// C ABI of the Ozaki-II-on-FP4 library (declarations and contracts in
// include/ozfp4.h). Host code: argument checks, per-device tables and
// workspace, kernel launches on the library stream, stage timing.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cstring>
#include <mutex>

#include "calibrate.hpp"
#include "karatsuba.hpp"
#include "kernels.hpp"
#include "onelimb.hpp"
#include "ozaki1.hpp"
#include "sgemm.hpp"
#include "split.hpp"
#include "ozfp4.h"
#include "tables.hpp"

using namespace ozfp4;

// Workspace of ozfp4_dgemm_noalloc (limb planes, residues, line maxima and
// the non-finite flag of one call): a fixed array in every device's copy of
// the code object, so that entry point never allocates. In host code this
// name is a host-side stand-in, not a device address: kernels and copies
// take the address hipGetSymbolAddress returns for the current device
// (DeviceState::scratch).
static __device__ __align__(256) uint8_t scratch[OZFP4_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
constexpr int kMaxStages = 8;

struct DeviceState {
  bool ready = false;
  ModConst* d_mod = nullptr;
  CrtConst* d_crt = nullptr;  // kMaxModuli + 1 entries, index L
  uint16_t* d_lut = nullptr;
  uint32_t* d_lut_k = nullptr;   // encoder LUT of the Karatsuba mode
  uint16_t* d_lut8 = nullptr;
  struct List {                 // a list with one-limb heads (index h)
    ModConst* mod = nullptr;
    ModConst* tail = nullptr;
    ModConst* head = nullptr;
    CrtConst* crt = nullptr;    // kMaxModuli + 1 entries, index L
    uint16_t* lut = nullptr;
  } lists[kMaxHeads + 1];
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
  int* h_flag = nullptr;      // pinned host word for the non-finite flag
  hipEvent_t ev[kMaxStages + 1] = {};
  uint8_t* scratch = nullptr; // this device's address of the scratch array
};

HostTables g_tables;
bool g_tables_ok = false;
std::once_flag g_tables_once;
DeviceState g_dev[kMaxDevices];
hipStream_t g_stream = nullptr;
bool g_profile = false;
bool g_karatsuba = false;
int g_heads = 0;             // one-limb heads of the scheme-II moduli list (0..kMaxHeads)
int g_cmax = 53;             // capacity cap: 53 (the paper's rule) .. 63
double g_stage_ms[kMaxStages];
int g_nstages = 0;
int g_pending_stages = 0;   // events recorded by the last profiled call
int g_pending_device = -1;

const HostTables* tables() {
  std::call_once(g_tables_once, [] { g_tables_ok = build_tables(g_tables); });
  return g_tables_ok ? &g_tables : nullptr;
}

inline int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

// Padded k of the limb planes: a multiple of the GEMM stage, at least
// kMinKPad (three stages).
inline int64_t plane_k_pad(int64_t k) {
  return std::max<int64_t>(kMinKPad, round_up(k, kStageK));
}

#define HIP_TRY(expr)                                  \
  do {                                                 \
    if ((expr) != hipSuccess) return OZFP4_EHIP;       \
  } while (0)

// Frees whatever the state holds (with its device current) and resets it.
void release_device(DeviceState& d) {
  (void)hipFree(d.ws);
  (void)hipFree(d.d_mod);
  (void)hipFree(d.d_crt);
  (void)hipFree(d.d_lut);
  (void)hipFree(d.d_lut_k);
  (void)hipFree(d.d_lut8);
  for (auto& Ld : d.lists) {
    (void)hipFree(Ld.mod);
    (void)hipFree(Ld.tail);
    (void)hipFree(Ld.head);
    (void)hipFree(Ld.crt);
    (void)hipFree(Ld.lut);
  }
  if (d.h_flag) (void)hipHostFree(d.h_flag);
  for (int e = 0; e <= kMaxStages; ++e)
    if (d.ev[e]) (void)hipEventDestroy(d.ev[e]);
  d = DeviceState();
}

int init_device(DeviceState& d, const HostTables* T) {
  HIP_TRY(hipMalloc(&d.d_mod, sizeof(ModConst)));
  HIP_TRY(hipMalloc(&d.d_crt, sizeof(CrtConst) * (kMaxModuli + 1)));
  HIP_TRY(hipMalloc(&d.d_lut, T->lut.size() * sizeof(uint16_t)));
  HIP_TRY(hipMalloc(&d.d_lut_k, T->lut_k.size() * sizeof(uint32_t)));
  HIP_TRY(hipMalloc(&d.d_lut8, sizeof(T->lut8)));
  HIP_TRY(hipMemcpy(d.d_mod, &T->mod, sizeof(ModConst), hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(d.d_crt, T->crt, sizeof(CrtConst) * (kMaxModuli + 1), hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(d.d_lut, T->lut.data(), T->lut.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(d.d_lut_k, T->lut_k.data(), T->lut_k.size() * sizeof(uint32_t),
                    hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(d.d_lut8, T->lut8, sizeof(T->lut8), hipMemcpyHostToDevice));
  for (int h = 1; h <= kMaxHeads; ++h) {
    const HostTables::List& Lh = T->lists[h];
    DeviceState::List& Ld = d.lists[h];
    HIP_TRY(hipMalloc(&Ld.mod, sizeof(ModConst)));
    HIP_TRY(hipMalloc(&Ld.tail, sizeof(ModConst)));
    HIP_TRY(hipMalloc(&Ld.head, sizeof(ModConst)));
    HIP_TRY(hipMalloc(&Ld.crt, sizeof(CrtConst) * (kMaxModuli + 1)));
    HIP_TRY(hipMalloc(&Ld.lut, Lh.lut.size() * sizeof(uint16_t)));
    HIP_TRY(hipMemcpy(Ld.mod, &Lh.mod, sizeof(ModConst), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(Ld.tail, &Lh.tail, sizeof(ModConst), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(Ld.head, &Lh.head, sizeof(ModConst), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(Ld.crt, Lh.crt, sizeof(CrtConst) * (kMaxModuli + 1), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(Ld.lut, Lh.lut.data(), Lh.lut.size() * sizeof(uint16_t),
                      hipMemcpyHostToDevice));
  }
  HIP_TRY(hipHostMalloc(reinterpret_cast<void**>(&d.h_flag), sizeof(int), hipHostMallocDefault));
  for (int i = 0; i <= kMaxStages; ++i) HIP_TRY(hipEventCreate(&d.ev[i]));
  // each device holds its own copy of the scratch array: keep its address
  void* sp = nullptr;
  HIP_TRY(hipGetSymbolAddress(&sp, HIP_SYMBOL(scratch)));
  if (!sp) return OZFP4_EHIP;
  d.scratch = static_cast<uint8_t*>(sp);
  return OZFP4_OK;
}

int device_state(DeviceState** out) {
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return OZFP4_EHIP;
  DeviceState& d = g_dev[dev];
  if (!d.ready) {
    if (init_device(d, T) != OZFP4_OK) {  // leave nothing half-made behind
      (void)hipGetLastError();
      release_device(d);
      return OZFP4_EHIP;
    }
    d.ready = true;
  }
  *out = &d;
  return OZFP4_OK;
}

int ensure_workspace(DeviceState* d, size_t bytes) {
  if (bytes <= d->ws_bytes) return OZFP4_OK;
  if (d->ws) {
    // an asynchronous call issued earlier on another stream may still use
    // the old buffer: wait for the whole device before freeing it
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipFree(d->ws));
    d->ws = nullptr;
    d->ws_bytes = 0;
  }
  size_t sz = (bytes + (size_t(1) << 20) - 1) & ~((size_t(1) << 20) - 1);
  if (hipMalloc(&d->ws, sz) != hipSuccess) {
    (void)hipGetLastError();
    return OZFP4_ENOMEM;
  }
  d->ws_bytes = sz;
  return OZFP4_OK;
}

// ---------------------------------------------------------------- plans

struct DgemmPlan {
  int64_t m, n, k;
  int L, cA, cB;
  int64_t m_pad, n_pad, k_pad, kblocks;
  int64_t plane_a, plane_b;  // bytes per plane
  bool kar;                  // Karatsuba mode
  bool f32;                  // FP32 inputs and output (capacity cap 24)
  int heads;                 // one-limb heads of the list (0: the greedy list)
  int nh;                    // of them among the call's L moduli: min(heads, L)
  int nplanes;               // planes per operand: 2L, plus the sum planes in the Karatsuba mode
  // workspace offsets
  size_t off_amax_a, off_amax_b, off_flag, off_pa, off_pb, off_r, total;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Each product of two dimensions at most OZFP4_MAX_ELEMENTS: then every
// padded size, plane, residue and partial-sum buffer fits in 64 bits.
bool dims_ok(int64_t m, int64_t n, int64_t k) {
  if (m < 0 || n < 0 || k < 0) return false;
  auto ok = [](int64_t a, int64_t b) { return a == 0 || b <= OZFP4_MAX_ELEMENTS / a; };
  return ok(m, n) && ok(m, k) && ok(n, k);
}

int check_dgemm_args(int64_t m, int64_t n, int64_t k, const void* A, int64_t lda, const void* B,
                     int64_t ldb, int n_moduli) {
  if (!dims_ok(m, n, k)) return OZFP4_EINVAL;
  if (lda < std::max<int64_t>(1, m) || ldb < std::max<int64_t>(1, k)) return OZFP4_EINVAL;
  if (n_moduli < OZFP4_MIN_MODULI || n_moduli > OZFP4_MAX_MODULI) return OZFP4_EMODULI;
  if (m > 0 && n > 0 && k > 0) {
    if (!A || !B) return OZFP4_EINVAL;
    if (k > OZFP4_MAX_K) return OZFP4_EKBOUND;
  }
  return OZFP4_OK;
}

// FP32 emulation: an FP32 significand's 24 bits in place of FP64's 53
constexpr int kFp32Capacity = 24;

int make_dgemm_plan(int64_t m, int64_t n, int64_t k, int L, DgemmPlan* p, bool f32 = false) {
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  p->m = m; p->n = n; p->k = k; p->L = L;
  p->f32 = f32;
  p->heads = g_heads;
  p->nh = std::min(g_heads, L);
  if (p->heads && g_karatsuba && !f32) return OZFP4_EINVAL;
  if (!capacity_split(p->heads ? T->lists[p->heads].P[L] : T->P[L], k,
                      f32 ? kFp32Capacity : g_cmax, &p->cA, &p->cB))
    return OZFP4_EMODULI;
  p->m_pad = round_up(m, kTile);
  p->n_pad = round_up(n, kTile);
  p->k_pad = plane_k_pad(k);
  p->kblocks = p->k_pad / kFragK;
  p->plane_a = p->m_pad * p->k_pad / 2;
  p->plane_b = p->n_pad * p->k_pad / 2;
  p->kar = g_karatsuba && !f32;
  p->nplanes = 2 * L + (p->kar ? T->nk[L] : 0);
  size_t off = 0;
  p->off_amax_a = off; off = align256(off + sizeof(uint64_t) * p->m_pad);
  p->off_amax_b = off; off = align256(off + sizeof(uint64_t) * p->n_pad);
  p->off_flag = off;   off = align256(off + 256);
  p->off_pa = off;     off = align256(off + (size_t)p->plane_a * p->nplanes);
  p->off_pb = off;     off = align256(off + (size_t)p->plane_b * p->nplanes);
  p->off_r = off;      off = align256(off + (size_t)p->m_pad * p->n_pad * L);
  p->total = off;
  return OZFP4_OK;
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// Stage times of an asynchronous profiled call (ozfp4_igemm_s8) are read
// from its events only when asked for; a later call records over the same
// events, so the pending times are read first.
int resolve_pending() {
  if (g_pending_stages <= 0) return OZFP4_OK;
  const int n = g_pending_stages;
  g_pending_stages = 0;
  DeviceState& d = g_dev[g_pending_device];
  HIP_TRY(hipEventSynchronize(d.ev[n]));
  for (int i = 0; i < n; ++i) {
    float t = 0.f;
    HIP_TRY(hipEventElapsedTime(&t, d.ev[i], d.ev[i + 1]));
    g_stage_ms[i] = t;
  }
  g_nstages = n;
  return OZFP4_OK;
}

void record(DeviceState* d, int i) {
  if (!g_profile) return;
  if (i == 0) (void)resolve_pending();   // before its events are recorded over
  (void)hipEventRecord(d->ev[i], g_stream);
}

int encode_grid(int64_t nfrag) {
  // enough blocks to fill the chip several times, each wave loops
  int64_t want = (nfrag + kEncWaves - 1) / kEncWaves;
  return (int)std::min<int64_t>(want, 256 * 16);
}

// Line maxima of the FP64 operands: rows of A (adjacent in memory) and
// columns of B (contiguous), one wave per column of B in launches of at
// most kLaunchThreads threads.
void launch_amax_f64(const double* A, int64_t lda, const double* B, int64_t ldb, int64_t m,
                     int64_t n, int64_t k, uint64_t* amax_a, uint64_t* amax_b, int* flag) {
  hipLaunchKernelGGL(k_amax_adjacent_lines, dim3(blocks_for(m, 256), blocks_for(k, kAmaxChunk)),
                     dim3(256), 0, g_stream, A, lda, m, k,
                     reinterpret_cast<unsigned long long*>(amax_a), flag);
  constexpr int64_t kLines = kLaunchThreads / 64;
  for (int64_t l0 = 0; l0 < n; l0 += kLines)
    hipLaunchKernelGGL(k_amax_contig_lines,
                       dim3(blocks_for(std::min(n - l0, kLines), 4), blocks_for(k, kAmaxContigChunk)),
                       dim3(256), 0, g_stream, B, ldb, n, k,
                       reinterpret_cast<unsigned long long*>(amax_b), flag, l0);
}

// Stages of the dgemm pipeline, stopping after `last`:
// 0 scale, 1 encode A, 2 encode B, 3 residue GEMM, 4 CRT.
// A, B and C are double, or float when p.f32.
int run_dgemm(const DgemmPlan& p, DeviceState* d, const void* Av, int64_t lda, const void* Bv,
              int64_t ldb, void* Cv, int64_t ldc, int last, uint8_t* planes_a_out,
              uint8_t* planes_b_out, uint8_t* ws_base = nullptr) {
  const double* A = static_cast<const double*>(Av);
  const double* B = static_cast<const double*>(Bv);
  const float* Af = static_cast<const float*>(Av);
  const float* Bf = static_cast<const float*>(Bv);
  const HostTables* T = tables();
  uint8_t* ws = ws_base ? ws_base : d->ws;
  uint64_t* amax_a = reinterpret_cast<uint64_t*>(ws + p.off_amax_a);
  uint64_t* amax_b = reinterpret_cast<uint64_t*>(ws + p.off_amax_b);
  int* flag = reinterpret_cast<int*>(ws + p.off_flag);
  uint8_t* pa = planes_a_out ? planes_a_out : ws + p.off_pa;
  uint8_t* pb = planes_b_out ? planes_b_out : ws + p.off_pb;
  uint8_t* R = ws + p.off_r;
  const int L = p.L;

  record(d, 0);
  // stage 0: line maxima (the flag word shares the zero fill)
  const int64_t nzero = (int64_t)((p.off_flag + 256 - p.off_amax_a) / sizeof(uint64_t));
  hipLaunchKernelGGL(k_fill_u64, dim3(blocks_for(nzero, 256)), dim3(256), 0, g_stream,
                     amax_a, nzero, (uint64_t)0);
  if (p.f32) {
    HIP_TRY(launch_amax_f32(g_stream, Af, lda, Bf, ldb, p.m, p.n, p.k, amax_a, amax_b, flag));
  } else {
    launch_amax_f64(A, lda, B, ldb, p.m, p.n, p.k, amax_a, amax_b, flag);
  }
  HIP_TRY(hipGetLastError());
  record(d, 1);
  if (last < 1) return OZFP4_OK;

  // stage 1, 2: fused conversion + residues + limbs + E2M1 packing
  const ModConst& mod = p.heads ? T->lists[p.heads].mod : T->mod;
  const ModConst* d_mod = p.heads ? d->lists[p.heads].mod : d->d_mod;
  const int lut_entries = mod.lut_off[L - 1] + 3 * mod.m[L - 1];
  const size_t lut_bytes = (p.kar ? sizeof(uint32_t) : sizeof(uint16_t)) * (size_t)lut_entries;
  const void* lut = p.kar ? static_cast<const void*>(d->d_lut_k)
                          : static_cast<const void*>(p.heads ? d->lists[p.heads].lut : d->d_lut);
  const int64_t nfa = (p.m_pad / kFragLines) * p.kblocks;
  const int64_t nfb = (p.n_pad / kFragLines) * p.kblocks;
  // an operand whose capacity exceeds 53 bits takes the wide encoder; the
  // Karatsuba mode's encoder lives in its own translation unit
  if (p.f32) {
    HIP_TRY(launch_encode_f32((unsigned)encode_grid(nfa), lut_bytes, g_stream, Af, (int64_t)1, lda,
                              p.m, p.k, amax_a, p.cA, pa, p.plane_a, nfa, p.kblocks, L, d_mod,
                              lut, lut_entries));
  } else if (p.kar) {
    HIP_TRY(launch_encode_kar(p.cA > 53, (unsigned)encode_grid(nfa), lut_bytes, g_stream, A,
                              (int64_t)1, lda, p.m, p.k, amax_a, p.cA, pa, p.plane_a, nfa,
                              p.kblocks, L, d->d_mod, lut, lut_entries));
  } else {
    auto enc = p.cA > 53 ? k_encode_dgemm<false, true> : k_encode_dgemm<false, false>;
    hipLaunchKernelGGL(enc,
                       dim3(encode_grid(nfa)), dim3(256), lut_bytes, g_stream, A, (int64_t)1, lda,
                       p.m, p.k, amax_a, p.cA, pa, p.plane_a, nfa, p.kblocks, L, d_mod, lut,
                       lut_entries, 0);
  }
  HIP_TRY(hipGetLastError());
  record(d, 2);
  if (p.f32) {
    HIP_TRY(launch_encode_f32((unsigned)encode_grid(nfb), lut_bytes, g_stream, Bf, ldb, (int64_t)1,
                              p.n, p.k, amax_b, p.cB, pb, p.plane_b, nfb, p.kblocks, L, d_mod,
                              lut, lut_entries));
  } else if (p.kar) {
    HIP_TRY(launch_encode_kar(p.cB > 53, (unsigned)encode_grid(nfb), lut_bytes, g_stream, B, ldb,
                              (int64_t)1, p.n, p.k, amax_b, p.cB, pb, p.plane_b, nfb, p.kblocks,
                              L, d->d_mod, lut, lut_entries));
  } else {
    auto enc = p.cB > 53 ? k_encode_dgemm<false, true> : k_encode_dgemm<false, false>;
    hipLaunchKernelGGL(enc,
                       dim3(encode_grid(nfb)), dim3(256), lut_bytes, g_stream, B, ldb, (int64_t)1,
                       p.n, p.k, amax_b, p.cB, pb, p.plane_b, nfb, p.kblocks, L, d_mod, lut,
                       lut_entries, 0);
  }
  HIP_TRY(hipGetLastError());
  record(d, 3);
  if (last < 3) return OZFP4_OK;

  // stage 3: fused residue GEMM for all moduli. In a list with one-limb
  // heads, the default GEMM covers the two-limb moduli after the heads from
  // their planes and residue planes on (with the list's tail constants),
  // and the heads take the single-product GEMM.
  const int64_t tiles_m = p.m_pad / kTileM, tiles_n = p.n_pad / kTileN;
  const int Lg = L - p.nh;
  const int64_t nblocks = tiles_m * tiles_n * Lg;
  const int64_t rplane = p.m_pad * p.n_pad;
  if (p.heads) {
    // the heads first: their short burst of residue writes then lands well
    // before the CRT reads
    HIP_TRY(launch_gemm_one_limb(g_stream, pa, pb, R, p.m_pad, rplane, p.plane_a, p.plane_b,
                                 p.m_pad, p.n_pad, p.kblocks, p.nh, d->lists[p.heads].head));
    if (Lg > 0) {
      hipLaunchKernelGGL(k_gemm_res, dim3((unsigned)nblocks), dim3(kWaves * 64), 0, g_stream,
                         pa + 2 * p.nh * p.plane_a, pb + 2 * p.nh * p.plane_b, R + p.nh * rplane,
                         p.plane_a, p.plane_b, p.kblocks, tiles_m, tiles_n, nblocks, p.m_pad,
                         rplane, d->lists[p.heads].tail);
      HIP_TRY(hipGetLastError());
    }
  } else if (p.kar) {
    HIP_TRY(launch_gemm_res_kar((unsigned)nblocks, g_stream, pa, pb, R, p.plane_a, p.plane_b,
                                p.kblocks, tiles_m, tiles_n, nblocks, p.m_pad, p.m_pad * p.n_pad,
                                d->d_mod, L));
  } else {
    hipLaunchKernelGGL(k_gemm_res, dim3((unsigned)nblocks), dim3(kWaves * 64), 0, g_stream, pa,
                       pb, R, p.plane_a, p.plane_b, p.kblocks, tiles_m, tiles_n, nblocks, p.m_pad,
                       p.m_pad * p.n_pad, d->d_mod);
  }
  HIP_TRY(hipGetLastError());
  record(d, 4);
  if (last < 4) return OZFP4_OK;

  // stage 4: CRT reconstruction and inverse scaling
  const int64_t nthreads = ((p.m + kCrtRows - 1) / kCrtRows) * p.n;
  const CrtConst* crt = (p.heads ? d->lists[p.heads].crt : d->d_crt) + L;
  const int nc = (p.heads ? T->lists[p.heads].crt : T->crt)[L].nc;
  if (p.f32) {
    HIP_TRY(launch_crt_f32(g_stream, nc, R, p.m_pad, rplane, p.m, p.n,
                           amax_a, amax_b, p.cA, p.cB, crt, static_cast<float*>(Cv),
                           ldc));
    record(d, 5);
    return OZFP4_OK;
  }
  double* C = static_cast<double*>(Cv);
  for (int64_t t0 = 0; t0 < nthreads; t0 += kLaunchThreads) {
    const unsigned grid = blocks_for(std::min(nthreads - t0, kLaunchThreads), 256);
    if (nc == 3)
      hipLaunchKernelGGL(k_crt<3>, dim3(grid), dim3(256), 0, g_stream, R, p.m_pad,
                         rplane, p.m, p.n, amax_a, amax_b, p.cA, p.cB, crt, C,
                         ldc, t0);
    else
      hipLaunchKernelGGL(k_crt<4>, dim3(grid), dim3(256), 0, g_stream, R, p.m_pad,
                         rplane, p.m, p.n, amax_a, amax_b, p.cA, p.cB, crt, C,
                         ldc, t0);
  }
  HIP_TRY(hipGetLastError());
  record(d, 5);
  return OZFP4_OK;
}

// ------------------------------------------------------- Ozaki scheme I

// c = floor(log2 min(X_p, 2^53)) with X_p = (13^p - 1) / 3 (Sec. IV-B)
int ozi_capacity_bits(int p) {
  uint64_t x = 1;
  for (int i = 0; i < p; ++i) x *= 13;
  x = std::min<uint64_t>((x - 1) / 3, uint64_t(1) << 53);
  return 63 - __builtin_clzll(x);
}

struct OziPlan {
  int64_t m, n, k;
  int p, nblk, nplanes, nh, cap;
  int64_t m_pad, n_pad, k_pad, kblocks;
  int64_t plane_a, plane_b;
  size_t off_amax_a, off_amax_b, off_flag, off_pa, off_pb, off_h, total;
};

int check_ozi_args(int64_t m, int64_t n, int64_t k, const void* A, int64_t lda, const void* B,
                   int64_t ldb, int n_limbs) {
  if (!dims_ok(m, n, k)) return OZFP4_EINVAL;
  if (lda < std::max<int64_t>(1, m) || ldb < std::max<int64_t>(1, k)) return OZFP4_EINVAL;
  if (n_limbs < 1 || n_limbs > OZFP4_OZI_MAX_LIMBS) return OZFP4_EINVAL;
  if (m > 0 && n > 0 && k > 0) {
    if (!A || !B) return OZFP4_EINVAL;
    if (k > OZFP4_MAX_K) return OZFP4_EKBOUND;
  }
  return OZFP4_OK;
}

void make_ozi_plan(int64_t m, int64_t n, int64_t k, int p, OziPlan* o) {
  o->m = m; o->n = n; o->k = k; o->p = p;
  o->nblk = (p + 2) / 3;
  o->nplanes = 3 * o->nblk;
  o->nh = 2 * o->nblk - 1;
  o->cap = ozi_capacity_bits(p);
  o->m_pad = round_up(m, kTile);
  o->n_pad = round_up(n, kTile);
  o->k_pad = plane_k_pad(k);
  o->kblocks = o->k_pad / kFragK;
  o->plane_a = o->m_pad * o->k_pad / 2;
  o->plane_b = o->n_pad * o->k_pad / 2;
  size_t off = 0;
  o->off_amax_a = off; off = align256(off + sizeof(uint64_t) * o->m_pad);
  o->off_amax_b = off; off = align256(off + sizeof(uint64_t) * o->n_pad);
  o->off_flag = off;   off = align256(off + 256);
  o->off_pa = off;     off = align256(off + (size_t)o->plane_a * o->nplanes);
  o->off_pb = off;     off = align256(off + (size_t)o->plane_b * o->nplanes);
  o->off_h = off;      off = align256(off + sizeof(int64_t) * (size_t)o->m_pad * o->n_pad * o->nh);
  o->total = off;
}

// Stages, stopping after `last`: 0 scale, 1 encode A, 2 encode B, 3 limb
// GEMM into the partial-sum planes, 4 reduction into C.
int run_ozi(const OziPlan& p, DeviceState* d, const double* A, int64_t lda, const double* B,
            int64_t ldb, double* C, int64_t ldc, int last, uint8_t* planes_a_out,
            uint8_t* planes_b_out) {
  uint8_t* ws = d->ws;
  uint64_t* amax_a = reinterpret_cast<uint64_t*>(ws + p.off_amax_a);
  uint64_t* amax_b = reinterpret_cast<uint64_t*>(ws + p.off_amax_b);
  int* flag = reinterpret_cast<int*>(ws + p.off_flag);
  uint8_t* pa = planes_a_out ? planes_a_out : ws + p.off_pa;
  uint8_t* pb = planes_b_out ? planes_b_out : ws + p.off_pb;
  int64_t* H = reinterpret_cast<int64_t*>(ws + p.off_h);

  record(d, 0);
  const int64_t nzero = (int64_t)((p.off_flag + 256 - p.off_amax_a) / sizeof(uint64_t));
  hipLaunchKernelGGL(k_fill_u64, dim3(blocks_for(nzero, 256)), dim3(256), 0, g_stream,
                     amax_a, nzero, (uint64_t)0);
  launch_amax_f64(A, lda, B, ldb, p.m, p.n, p.k, amax_a, amax_b, flag);
  HIP_TRY(hipGetLastError());
  record(d, 1);
  if (last < 1) return OZFP4_OK;

  const int64_t nfa = (p.m_pad / kFragLines) * p.kblocks;
  const int64_t nfb = (p.n_pad / kFragLines) * p.kblocks;
  HIP_TRY(launch_encode_ozi((unsigned)encode_grid(nfa), g_stream, A, (int64_t)1, lda, p.m, p.k,
                            amax_a, p.cap, pa, p.plane_a, nfa, p.kblocks, p.nplanes));
  record(d, 2);
  HIP_TRY(launch_encode_ozi((unsigned)encode_grid(nfb), g_stream, B, ldb, (int64_t)1, p.n, p.k,
                            amax_b, p.cap, pb, p.plane_b, nfb, p.kblocks, p.nplanes));
  record(d, 3);
  if (last < 3) return OZFP4_OK;

  HIP_TRY(launch_gemm_ozi(g_stream, pa, pb, H, p.plane_a, p.plane_b, p.kblocks, p.m_pad, p.n_pad,
                          p.nblk));
  record(d, 4);
  if (last < 4) return OZFP4_OK;

  HIP_TRY(launch_ozi_reduce(g_stream, H, p.m_pad, p.m_pad * p.n_pad, p.nh, p.m, p.n, amax_a,
                            amax_b, p.cap, C, ldc));
  record(d, 5);
  return OZFP4_OK;
}

int prepare_ozi(int64_t m, int64_t n, int64_t k, int n_limbs, OziPlan* p, DeviceState** d) {
  make_ozi_plan(m, n, k, n_limbs, p);
  int rc = device_state(d);
  if (rc) return rc;
  return ensure_workspace(*d, p->total);
}

int finish_with_flag(DeviceState* d, const int* dflag, int nstages) {
  HIP_TRY(hipMemcpyAsync(d->h_flag, dflag, sizeof(int), hipMemcpyDeviceToHost, g_stream));
  HIP_TRY(hipStreamSynchronize(g_stream));
  if (g_profile && nstages > 0) {
    g_pending_stages = 0;
    for (int i = 0; i < nstages; ++i) {
      float ms = 0.f;
      HIP_TRY(hipEventElapsedTime(&ms, d->ev[i], d->ev[i + 1]));
      g_stage_ms[i] = ms;
    }
    g_nstages = nstages;
  }
  return *d->h_flag ? OZFP4_ENONFINITE : OZFP4_OK;
}

// ------------------------------------------------------ two-term split

// The split route: the paper's 53-bit capacities for both terms, d =
// min(c_A, c_B); four planes sets (A1, A2, B1, B2) and four residue sets.
struct SplitPlan {
  int64_t m, n, k;
  int L, cA, cB, d;
  int heads, nh;             // one-limb heads of the list, and of them among the L moduli
  int64_t m_pad, n_pad, k_pad, kblocks, plane_a, plane_b, rset;
  size_t off_amax_a, off_amax_b, off_flag, off_pa1, off_pa2, off_pb1, off_pb2, off_r, total;
};

int make_split_plan(int64_t m, int64_t n, int64_t k, int L, SplitPlan* p) {
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  p->m = m; p->n = n; p->k = k; p->L = L;
  p->heads = g_heads;
  p->nh = std::min(g_heads, L);
  if (!capacity_split(p->heads ? T->lists[p->heads].P[L] : T->P[L], k, 53, &p->cA, &p->cB))
    return OZFP4_EMODULI;
  p->d = std::min(p->cA, p->cB);
  p->m_pad = round_up(m, kTile);
  p->n_pad = round_up(n, kTile);
  p->k_pad = plane_k_pad(k);
  p->kblocks = p->k_pad / kFragK;
  p->plane_a = p->m_pad * p->k_pad / 2;
  p->plane_b = p->n_pad * p->k_pad / 2;
  p->rset = p->m_pad * p->n_pad * L;
  size_t off = 0;
  p->off_amax_a = off; off = align256(off + sizeof(uint64_t) * p->m_pad);
  p->off_amax_b = off; off = align256(off + sizeof(uint64_t) * p->n_pad);
  p->off_flag = off;   off = align256(off + 256);
  p->off_pa1 = off;    off = align256(off + (size_t)p->plane_a * 2 * L);
  p->off_pa2 = off;    off = align256(off + (size_t)p->plane_a * 2 * L);
  p->off_pb1 = off;    off = align256(off + (size_t)p->plane_b * 2 * L);
  p->off_pb2 = off;    off = align256(off + (size_t)p->plane_b * 2 * L);
  p->off_r = off;      off = align256(off + (size_t)p->rset * 4);
  p->total = off;
  return OZFP4_OK;
}

// Stages: 0 scale, 1 encode A (both terms), 2 encode B (both terms), 3 the
// four residue GEMMs, 4 the combined CRT.
int run_split(const SplitPlan& p, DeviceState* d, const double* A, int64_t lda, const double* B,
              int64_t ldb, double* C, int64_t ldc) {
  const HostTables* T = tables();
  uint8_t* ws = d->ws;
  uint64_t* amax_a = reinterpret_cast<uint64_t*>(ws + p.off_amax_a);
  uint64_t* amax_b = reinterpret_cast<uint64_t*>(ws + p.off_amax_b);
  int* flag = reinterpret_cast<int*>(ws + p.off_flag);
  const int L = p.L;
  record(d, 0);
  const int64_t nzero = (int64_t)((p.off_flag + 256 - p.off_amax_a) / sizeof(uint64_t));
  hipLaunchKernelGGL(k_fill_u64, dim3(blocks_for(nzero, 256)), dim3(256), 0, g_stream, amax_a,
                     nzero, (uint64_t)0);
  launch_amax_f64(A, lda, B, ldb, p.m, p.n, p.k, amax_a, amax_b, flag);
  HIP_TRY(hipGetLastError());
  record(d, 1);
  // the moduli list: the greedy one, or one with one-limb heads
  const ModConst& mod = p.heads ? T->lists[p.heads].mod : T->mod;
  const ModConst* d_mod = p.heads ? d->lists[p.heads].mod : d->d_mod;
  const uint16_t* d_lut = p.heads ? d->lists[p.heads].lut : d->d_lut;
  const int lut_entries = mod.lut_off[L - 1] + 3 * mod.m[L - 1];
  const size_t lut_bytes = sizeof(uint16_t) * (size_t)lut_entries;
  const int64_t nfa = (p.m_pad / kFragLines) * p.kblocks;
  const int64_t nfb = (p.n_pad / kFragLines) * p.kblocks;
  for (int term = 0; term < 2; ++term)
    HIP_TRY(launch_encode_split(term == 1, false, (unsigned)encode_grid(nfa), lut_bytes, g_stream, A,
                                (int64_t)1, lda, p.m, p.k, amax_a, p.cA,
                                ws + (term ? p.off_pa2 : p.off_pa1), p.plane_a, nfa, p.kblocks, L,
                                d_mod, d_lut, lut_entries, p.d));
  record(d, 2);
  for (int term = 0; term < 2; ++term)
    HIP_TRY(launch_encode_split(term == 1, false, (unsigned)encode_grid(nfb), lut_bytes, g_stream, B,
                                ldb, (int64_t)1, p.n, p.k, amax_b, p.cB,
                                ws + (term ? p.off_pb2 : p.off_pb1), p.plane_b, nfb, p.kblocks, L,
                                d_mod, d_lut, lut_entries, p.d));
  record(d, 3);
  // residue sets: A1 B1, A1 B2, A2 B1, A2 B2; with heads, the heads by the
  // single-product GEMM, then the two-limb moduli from their planes on
  const int64_t tiles_m = p.m_pad / kTileM, tiles_n = p.n_pad / kTileN;
  const int Lg = L - p.nh;
  const int64_t nblocks = tiles_m * tiles_n * Lg;
  const int64_t rplane = p.m_pad * p.n_pad;
  const size_t pa[4] = {p.off_pa1, p.off_pa1, p.off_pa2, p.off_pa2};
  const size_t pb[4] = {p.off_pb1, p.off_pb2, p.off_pb1, p.off_pb2};
  const ModConst* d_tail = p.heads ? d->lists[p.heads].tail : d->d_mod;
  for (int q = 0; q < 4; ++q) {
    uint8_t* Rq = ws + p.off_r + (size_t)q * p.rset;
    if (p.heads)
      HIP_TRY(launch_gemm_one_limb(g_stream, ws + pa[q], ws + pb[q], Rq, p.m_pad, rplane,
                                   p.plane_a, p.plane_b, p.m_pad, p.n_pad, p.kblocks, p.nh,
                                   d->lists[p.heads].head));
    if (Lg > 0)
      hipLaunchKernelGGL(k_gemm_res, dim3((unsigned)nblocks), dim3(kWaves * 64), 0, g_stream,
                         ws + pa[q] + 2 * p.nh * p.plane_a, ws + pb[q] + 2 * p.nh * p.plane_b,
                         Rq + p.nh * rplane, p.plane_a, p.plane_b, p.kblocks, tiles_m, tiles_n,
                         nblocks, p.m_pad, rplane, d_tail);
  }
  HIP_TRY(hipGetLastError());
  record(d, 4);
  const uint8_t* R = ws + p.off_r;
  const int nc = (p.heads ? T->lists[p.heads].crt : T->crt)[L].nc;
  const CrtConst* crt = (p.heads ? d->lists[p.heads].crt : d->d_crt) + L;
  HIP_TRY(launch_crt_split(g_stream, nc, R, R + p.rset, R + 2 * p.rset, R + 3 * p.rset,
                           p.m_pad, rplane, p.m, p.n, amax_a, amax_b, p.cA, p.cB, p.d,
                           d_mod, crt, C, ldc));
  record(d, 5);
  return OZFP4_OK;
}

int prepare(int64_t m, int64_t n, int64_t k, int L, DgemmPlan* p, DeviceState** d,
            bool f32 = false) {
  int rc = make_dgemm_plan(m, n, k, L, p, f32);
  if (rc) return rc;
  rc = device_state(d);
  if (rc) return rc;
  return ensure_workspace(*d, p->total);
}

}  // namespace

extern "C" {

int ozfp4_dgemm(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda, const double* B,
                int64_t ldb, double* C, int64_t ldc, int n_moduli) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (ldc < std::max<int64_t>(1, m)) return OZFP4_EINVAL;
  if (m == 0 || n == 0) return OZFP4_OK;
  if (!C) return OZFP4_EINVAL;
  if (k == 0) {
    DeviceState* d;
    rc = device_state(&d);
    if (rc) return rc;
    hipLaunchKernelGGL(k_fill_f64_matrix, dim3(stride_blocks(m * n, 256)), dim3(256), 0, g_stream, C,
                       m, n, ldc);
    HIP_TRY(hipGetLastError());
    return OZFP4_OK;
  }
  DgemmPlan p;
  DeviceState* d;
  rc = prepare(m, n, k, n_moduli, &p, &d);
  if (rc) return rc;
  rc = run_dgemm(p, d, A, lda, B, ldb, C, ldc, 4, nullptr, nullptr);
  if (rc) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 5);
}

int ozfp4_init(void) {
  DeviceState* d;
  return device_state(&d);
}

int ozfp4_dgemm_noalloc(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                        const double* B, int64_t ldb, double* C, int64_t ldc, int n_moduli) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (ldc < std::max<int64_t>(1, m)) return OZFP4_EINVAL;
  if (m == 0 || n == 0) return OZFP4_OK;
  if (!C) return OZFP4_EINVAL;
  // the device must have been set up (ozfp4_init or any earlier call on
  // it): setting up allocates, and this entry point must not
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices || !g_dev[dev].ready || !tables()) return OZFP4_ESCRATCH;
  DeviceState* d = &g_dev[dev];
  if (k == 0) {
    hipLaunchKernelGGL(k_fill_f64_matrix, dim3(stride_blocks(m * n, 256)), dim3(256), 0, g_stream, C,
                       m, n, ldc);
    HIP_TRY(hipGetLastError());
    return OZFP4_OK;
  }
  DgemmPlan p;
  rc = make_dgemm_plan(m, n, k, n_moduli, &p);
  if (rc) return rc;
  if (p.total > (size_t)OZFP4_SCRATCH_BYTES) return OZFP4_ESCRATCH;
  // under stream capture the kernels are recorded into the caller's graph:
  // no stage events, and no read-back of the non-finite flag (that would
  // synchronize the capturing stream)
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  HIP_TRY(hipStreamIsCapturing(g_stream, &capture));
  const bool captured = capture != hipStreamCaptureStatusNone;
  const bool profile = g_profile;
  if (captured) g_profile = false;
  rc = run_dgemm(p, d, A, lda, B, ldb, C, ldc, 4, nullptr, nullptr, d->scratch);
  g_profile = profile;
  if (rc || captured) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->scratch + p.off_flag), 5);
}

int ozfp4_dgemm_split(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                      const double* B, int64_t ldb, double* C, int64_t ldc, int n_moduli) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (ldc < std::max<int64_t>(1, m)) return OZFP4_EINVAL;
  if (m == 0 || n == 0) return OZFP4_OK;
  if (!C) return OZFP4_EINVAL;
  DeviceState* d;
  if (k == 0) {
    rc = device_state(&d);
    if (rc) return rc;
    hipLaunchKernelGGL(k_fill_f64_matrix, dim3(stride_blocks(m * n, 256)), dim3(256), 0, g_stream, C,
                       m, n, ldc);
    HIP_TRY(hipGetLastError());
    return OZFP4_OK;
  }
  SplitPlan p;
  rc = make_split_plan(m, n, k, n_moduli, &p);
  if (rc) return rc;
  rc = device_state(&d);
  if (rc) return rc;
  rc = ensure_workspace(d, p.total);
  if (rc) return rc;
  rc = run_split(p, d, A, lda, B, ldb, C, ldc);
  if (rc) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 5);
}

int ozfp4_igemm_s8(int64_t m, int64_t n, int64_t k, const int8_t* A, int64_t lda, const int8_t* B,
                   int64_t ldb, int32_t* C, int64_t ldc) {
  if (!dims_ok(m, n, k)) return OZFP4_EINVAL;
  if (lda < std::max<int64_t>(1, m) || ldb < std::max<int64_t>(1, k) ||
      ldc < std::max<int64_t>(1, m))
    return OZFP4_EINVAL;
  if (m == 0 || n == 0) return OZFP4_OK;
  if (!C) return OZFP4_EINVAL;
  if (k > OZFP4_MAX_K_S8) return OZFP4_EKBOUND;
  DeviceState* d;
  int rc = device_state(&d);
  if (rc) return rc;
  if (k == 0) {
    hipLaunchKernelGGL(k_fill_i32_matrix, dim3(stride_blocks(m * n, 256)), dim3(256), 0, g_stream, C,
                       m, n, ldc);
    HIP_TRY(hipGetLastError());
    return OZFP4_OK;
  }
  if (!A || !B) return OZFP4_EINVAL;
  const int64_t m_pad = round_up(m, kTile), n_pad = round_up(n, kTile);
  const int64_t k_pad = plane_k_pad(k), kblocks = k_pad / kFragK;
  const int64_t plane_a = m_pad * k_pad / 2, plane_b = n_pad * k_pad / 2;
  const size_t off_pb = align256((size_t)plane_a * 3);
  rc = ensure_workspace(d, off_pb + align256((size_t)plane_b * 3));
  if (rc) return rc;
  uint8_t* pa = d->ws;
  uint8_t* pb = d->ws + off_pb;
  record(d, 0);
  const int64_t nfa = (m_pad / kFragLines) * kblocks, nfb = (n_pad / kFragLines) * kblocks;
  hipLaunchKernelGGL(k_encode_s8, dim3(encode_grid(nfa)), dim3(256), 0, g_stream, A, (int64_t)1,
                     lda, m, k, pa, plane_a, nfa, kblocks, d->d_lut8);
  record(d, 1);
  hipLaunchKernelGGL(k_encode_s8, dim3(encode_grid(nfb)), dim3(256), 0, g_stream, B, ldb,
                     (int64_t)1, n, k, pb, plane_b, nfb, kblocks, d->d_lut8);
  record(d, 2);
  const int64_t tiles_m = m_pad / kTileS8M, tiles_n = n_pad / kTileS8N;
  const int64_t nblocks = tiles_m * tiles_n;
  hipLaunchKernelGGL(k_gemm_s8, dim3((unsigned)nblocks), dim3(kWaves * 64), 0, g_stream, pa, pb, C,
                     plane_a, plane_b, kblocks, tiles_m, tiles_n, nblocks, m, n, ldc);
  record(d, 3);
  HIP_TRY(hipGetLastError());
  if (g_profile) {
    g_pending_stages = 3;
    HIP_TRY(hipGetDevice(&g_pending_device));
  }
  return OZFP4_OK;
}

int ozfp4_sgemm(int64_t m, int64_t n, int64_t k, const float* A, int64_t lda, const float* B,
                int64_t ldb, float* C, int64_t ldc, int n_moduli) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (ldc < std::max<int64_t>(1, m)) return OZFP4_EINVAL;
  if (m == 0 || n == 0) return OZFP4_OK;
  if (!C) return OZFP4_EINVAL;
  if (k == 0) {
    DeviceState* d;
    rc = device_state(&d);
    if (rc) return rc;
    // +0.0f has the bit pattern of the int32 zero
    hipLaunchKernelGGL(k_fill_i32_matrix, dim3(stride_blocks(m * n, 256)), dim3(256), 0, g_stream,
                       reinterpret_cast<int32_t*>(C), m, n, ldc);
    HIP_TRY(hipGetLastError());
    return OZFP4_OK;
  }
  DgemmPlan p;
  DeviceState* d;
  rc = prepare(m, n, k, n_moduli, &p, &d, true);
  if (rc) return rc;
  rc = run_dgemm(p, d, A, lda, B, ldb, C, ldc, 4, nullptr, nullptr);
  if (rc) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 5);
}

int ozfp4_sgemm_capacity(int64_t k, int n_moduli, int32_t* c_a, int32_t* c_b) {
  if (k < 1 || !c_a || !c_b) return OZFP4_EINVAL;
  if (n_moduli < OZFP4_MIN_MODULI || n_moduli > OZFP4_MAX_MODULI) return OZFP4_EMODULI;
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  int a, b;
  if (!capacity_split(g_heads ? T->lists[g_heads].P[n_moduli] : T->P[n_moduli], k, kFp32Capacity,
                      &a, &b))
    return OZFP4_EMODULI;
  *c_a = a;
  *c_b = b;
  return OZFP4_OK;
}

int ozfp4_dgemm_ozi(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                    const double* B, int64_t ldb, double* C, int64_t ldc, int n_limbs) {
  int rc = check_ozi_args(m, n, k, A, lda, B, ldb, n_limbs);
  if (rc) return rc;
  if (ldc < std::max<int64_t>(1, m)) return OZFP4_EINVAL;
  if (m == 0 || n == 0) return OZFP4_OK;
  if (!C) return OZFP4_EINVAL;
  if (k == 0) {
    DeviceState* d;
    rc = device_state(&d);
    if (rc) return rc;
    hipLaunchKernelGGL(k_fill_f64_matrix, dim3(stride_blocks(m * n, 256)), dim3(256), 0, g_stream, C,
                       m, n, ldc);
    HIP_TRY(hipGetLastError());
    return OZFP4_OK;
  }
  OziPlan p;
  DeviceState* d;
  rc = prepare_ozi(m, n, k, n_limbs, &p, &d);
  if (rc) return rc;
  rc = run_ozi(p, d, A, lda, B, ldb, C, ldc, 4, nullptr, nullptr);
  if (rc) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 5);
}

int ozfp4_ozi_config(int n_limbs, int32_t* capacity, int32_t* n_planes, int32_t* n_groups) {
  if (n_limbs < 1 || n_limbs > OZFP4_OZI_MAX_LIMBS) return OZFP4_EINVAL;
  const int nblk = (n_limbs + 2) / 3;
  if (capacity) *capacity = ozi_capacity_bits(n_limbs);
  if (n_planes) *n_planes = 3 * nblk;
  if (n_groups) *n_groups = 2 * nblk - 1;
  return OZFP4_OK;
}

int ozfp4_ozi_limb_planes(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                          const double* B, int64_t ldb, int n_limbs, uint8_t* planes_a,
                          uint8_t* planes_b) {
  int rc = check_ozi_args(m, n, k, A, lda, B, ldb, n_limbs);
  if (rc) return rc;
  if (m == 0 || n == 0 || k == 0) return OZFP4_EINVAL;
  if (!planes_a || !planes_b) return OZFP4_EINVAL;
  OziPlan p;
  DeviceState* d;
  rc = prepare_ozi(m, n, k, n_limbs, &p, &d);
  if (rc) return rc;
  rc = run_ozi(p, d, A, lda, B, ldb, nullptr, 0, 2, planes_a, planes_b);
  if (rc) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 0);
}

int ozfp4_ozi_partials(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                       const double* B, int64_t ldb, int n_limbs, int64_t* H, int64_t ldh) {
  int rc = check_ozi_args(m, n, k, A, lda, B, ldb, n_limbs);
  if (rc) return rc;
  if (m == 0 || n == 0 || k == 0) return OZFP4_EINVAL;
  if (!H || ldh < m) return OZFP4_EINVAL;
  OziPlan p;
  DeviceState* d;
  rc = prepare_ozi(m, n, k, n_limbs, &p, &d);
  if (rc) return rc;
  rc = run_ozi(p, d, A, lda, B, ldb, nullptr, 0, 3, nullptr, nullptr);
  if (rc) return rc;
  for (int h = 0; h < p.nh; ++h) {
    HIP_TRY(hipMemcpy2DAsync(H + (size_t)h * ldh * n, (size_t)ldh * sizeof(int64_t),
                             d->ws + p.off_h + (size_t)h * p.m_pad * p.n_pad * sizeof(int64_t),
                             (size_t)p.m_pad * sizeof(int64_t), (size_t)m * sizeof(int64_t),
                             (size_t)n, hipMemcpyDeviceToDevice, g_stream));
  }
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 0);
}

int ozfp4_set_stream(void* stream) {
  g_stream = reinterpret_cast<hipStream_t>(stream);
  return OZFP4_OK;
}

int ozfp4_finalize(void) {
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) cur = -1;
  for (int i = 0; i < kMaxDevices; ++i) {
    DeviceState& d = g_dev[i];
    if (!d.ready) continue;
    if (hipSetDevice(i) != hipSuccess) continue;
    (void)hipDeviceSynchronize();
    release_device(d);
  }
  // the events of a pending profiled call are gone with the device state
  g_pending_stages = 0;
  g_nstages = 0;
  if (cur >= 0) (void)hipSetDevice(cur);
  return OZFP4_OK;
}

const char* ozfp4_strerror(int code) {
  switch (code) {
    case OZFP4_OK: return "success";
    case OZFP4_EINVAL: return "invalid size, leading dimension or null pointer";
    case OZFP4_EMODULI: return "n_moduli outside [2, 27] or too few moduli for this k";
    case OZFP4_EKBOUND: return "k above the FP32-exactness bound";
    case OZFP4_ENONFINITE: return "NaN or Inf in an input matrix";
    case OZFP4_ENOMEM: return "device workspace allocation failed";
    case OZFP4_EHIP: return "HIP runtime error";
    case OZFP4_ESCRATCH:
      return "ozfp4_dgemm_noalloc: device not set up (call ozfp4_init), or the call needs more "
             "scratch than OZFP4_SCRATCH_BYTES";
    default: return "unknown error code";
  }
}

int ozfp4_moduli(int n_moduli, int32_t* out) {
  if (n_moduli < 1 || n_moduli > OZFP4_MAX_MODULI || !out) return OZFP4_EINVAL;
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  const std::vector<int>& list = g_heads ? T->lists[g_heads].moduli : T->moduli;
  for (int i = 0; i < n_moduli; ++i) out[i] = list[i];
  return OZFP4_OK;
}

int ozfp4_capacity(int64_t k, int n_moduli, int32_t* c_a, int32_t* c_b) {
  if (k < 1 || !c_a || !c_b) return OZFP4_EINVAL;
  if (n_moduli < OZFP4_MIN_MODULI || n_moduli > OZFP4_MAX_MODULI) return OZFP4_EMODULI;
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  int a, b;
  if (!capacity_split(g_heads ? T->lists[g_heads].P[n_moduli] : T->P[n_moduli], k, g_cmax, &a, &b))
    return OZFP4_EMODULI;
  *c_a = a;
  *c_b = b;
  return OZFP4_OK;
}

int ozfp4_two_limb_table(int modulus_index, uint8_t* out, int32_t* m_out) {
  if (modulus_index < 0 || modulus_index >= OZFP4_MAX_MODULI || !out || !m_out) return OZFP4_EINVAL;
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  const ModConst& mod = g_heads ? T->lists[g_heads].mod : T->mod;
  const int m = mod.m[modulus_index];
  const uint16_t* lut = (g_heads ? T->lists[g_heads].lut.data() : T->lut.data()) + mod.lut_off[modulus_index];
  for (int r = 0; r < m; ++r) {
    const uint16_t e = lut[r + m];  // remainder estimate r, non-negative value
    out[r] = (uint8_t)((e & 0xf) | ((e >> 8) & 0xf) << 4);
  }
  *m_out = m;
  return OZFP4_OK;
}

int ozfp4_sum_limb_table(int modulus_index, uint8_t* out, int32_t* m_out) {
  if (modulus_index < 0 || modulus_index >= OZFP4_MAX_MODULI || !out || !m_out) return OZFP4_EINVAL;
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  if (T->mod.ksum[modulus_index] < 0) return OZFP4_EINVAL;
  const int m = T->moduli[modulus_index];
  const uint32_t* lut = T->lut_k.data() + T->mod.lut_off[modulus_index];
  for (int r = 0; r < m; ++r) {
    const uint32_t e = lut[r + m];  // entry of the remainder estimate r itself
    out[r] = (uint8_t)((e & 0xf) | ((e >> 8) & 0xf) << 4);
  }
  *m_out = m;
  return OZFP4_OK;
}

int ozfp4_set_karatsuba(int enable) {
  g_karatsuba = enable != 0;
  return OZFP4_OK;
}

int ozfp4_set_one_limb_moduli(int heads) {
  if (heads < 0 || heads > kMaxHeads) return OZFP4_EINVAL;
  g_heads = heads;
  return OZFP4_OK;
}

int ozfp4_set_max_capacity(int bits) {
  if (bits < 53 || bits > 63) return OZFP4_EINVAL;
  g_cmax = bits;
  return OZFP4_OK;
}

int ozfp4_plane_count(int n_moduli, int32_t* n_planes, int32_t* sum_plane) {
  if (n_moduli < OZFP4_MIN_MODULI || n_moduli > OZFP4_MAX_MODULI) return OZFP4_EMODULI;
  if (!n_planes) return OZFP4_EINVAL;
  const HostTables* T = tables();
  if (!T) return OZFP4_EHIP;
  if (g_karatsuba && g_heads) return OZFP4_EINVAL;
  *n_planes = 2 * n_moduli + (g_karatsuba ? T->nk[n_moduli] : 0);
  if (sum_plane)
    for (int l = 0; l < n_moduli; ++l)
      sum_plane[l] = (g_karatsuba && T->mod.ksum[l] >= 0) ? 2 * n_moduli + T->mod.ksum[l] : -1;
  return OZFP4_OK;
}

int ozfp4_plane_layout(int64_t lines, int64_t k, int64_t* rows_pad, int64_t* k_pad,
                       int64_t* bytes_per_plane) {
  if (!dims_ok(lines, 0, k) || !rows_pad || !k_pad || !bytes_per_plane) return OZFP4_EINVAL;
  *rows_pad = round_up(lines, kTile);
  *k_pad = plane_k_pad(k);
  *bytes_per_plane = *rows_pad * *k_pad / 2;
  return OZFP4_OK;
}

int ozfp4_scales(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda, const double* B,
                 int64_t ldb, int n_moduli, int32_t* s, int32_t* t) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (m == 0 || n == 0 || k == 0) return OZFP4_EINVAL;
  if (!s || !t) return OZFP4_EINVAL;
  DgemmPlan p;
  DeviceState* d;
  rc = prepare(m, n, k, n_moduli, &p, &d);
  if (rc) return rc;
  rc = run_dgemm(p, d, A, lda, B, ldb, nullptr, 0, 0, nullptr, nullptr);
  if (rc) return rc;
  hipLaunchKernelGGL(k_shifts, dim3(blocks_for(m, 256)), dim3(256), 0, g_stream,
                     reinterpret_cast<uint64_t*>(d->ws + p.off_amax_a), m, p.cA, s);
  hipLaunchKernelGGL(k_shifts, dim3(blocks_for(n, 256)), dim3(256), 0, g_stream,
                     reinterpret_cast<uint64_t*>(d->ws + p.off_amax_b), n, p.cB, t);
  HIP_TRY(hipGetLastError());
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 0);
}

int ozfp4_limb_planes(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda,
                      const double* B, int64_t ldb, int n_moduli, uint8_t* planes_a,
                      uint8_t* planes_b) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (m == 0 || n == 0 || k == 0) return OZFP4_EINVAL;
  if (!planes_a || !planes_b) return OZFP4_EINVAL;
  DgemmPlan p;
  DeviceState* d;
  rc = prepare(m, n, k, n_moduli, &p, &d);
  if (rc) return rc;
  rc = run_dgemm(p, d, A, lda, B, ldb, nullptr, 0, 2, planes_a, planes_b);
  if (rc) return rc;
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 0);
}

int ozfp4_residues(int64_t m, int64_t n, int64_t k, const double* A, int64_t lda, const double* B,
                   int64_t ldb, int n_moduli, uint8_t* R, int64_t ldr) {
  int rc = check_dgemm_args(m, n, k, A, lda, B, ldb, n_moduli);
  if (rc) return rc;
  if (m == 0 || n == 0 || k == 0) return OZFP4_EINVAL;
  if (!R || ldr < m) return OZFP4_EINVAL;
  DgemmPlan p;
  DeviceState* d;
  rc = prepare(m, n, k, n_moduli, &p, &d);
  if (rc) return rc;
  rc = run_dgemm(p, d, A, lda, B, ldb, nullptr, 0, 3, nullptr, nullptr);
  if (rc) return rc;
  for (int l = 0; l < n_moduli; ++l) {
    HIP_TRY(hipMemcpy2DAsync(R + (size_t)l * ldr * n, (size_t)ldr,
                             d->ws + p.off_r + (size_t)l * p.m_pad * p.n_pad, (size_t)p.m_pad,
                             (size_t)m, (size_t)n, hipMemcpyDeviceToDevice, g_stream));
  }
  return finish_with_flag(d, reinterpret_cast<int*>(d->ws + p.off_flag), 0);
}

int ozfp4_calib_mfma(int64_t blocks, int64_t iterations, uint32_t seed, float* sink) {
  if (blocks < 1 || blocks > (int64_t(1) << 22) || iterations < 1 || !sink) return OZFP4_EINVAL;
  HIP_TRY(launch_calib_mfma(g_stream, blocks, iterations, seed, sink));
  return OZFP4_OK;
}

int ozfp4_calib_mfma_codes(int64_t blocks, int64_t iterations, const uint32_t* codes_a,
                           const uint32_t* codes_b, int64_t nwords, float* sink) {
  if (blocks < 1 || blocks > (int64_t(1) << 22) || iterations < 1 || !sink) return OZFP4_EINVAL;
  if (!codes_a || !codes_b || nwords < 16 || nwords % 16) return OZFP4_EINVAL;
  HIP_TRY(launch_calib_mfma_codes(g_stream, blocks, iterations, codes_a, codes_b, nwords, sink));
  return OZFP4_OK;
}

int ozfp4_calib_gemm_fp4(int64_t m, int64_t n, int64_t k, const uint8_t* plane_a,
                         const uint8_t* plane_b, float* C, int64_t ldc) {
  if (m < kTile || n < kTile || m % kTile || n % kTile || !dims_ok(m, n, k)) return OZFP4_EINVAL;
  if (k < kMinKPad || k % kStageK || k > 65536) return OZFP4_EINVAL;
  if ((m / kTile) * (n / kTile) > (int64_t(1) << 31) - 1) return OZFP4_EINVAL;
  if (!plane_a || !plane_b || !C || ldc < m) return OZFP4_EINVAL;
  HIP_TRY(launch_calib_gemm_fp4(g_stream, m, n, k, plane_a, plane_b, C, ldc));
  return OZFP4_OK;
}

int ozfp4_calib_dma_read(const uint8_t* src, int64_t bytes, int64_t blocks, uint32_t* sink) {
  if (bytes < kFragBytes || bytes % kFragBytes || bytes > (int64_t(1) << 31) - kFragBytes)
    return OZFP4_EINVAL;
  if (blocks < 1 || blocks > (int64_t(1) << 22) || !src || !sink) return OZFP4_EINVAL;
  HIP_TRY(launch_calib_dma_read(g_stream, src, bytes, blocks, sink));
  return OZFP4_OK;
}

int ozfp4_profile(int enable) {
  g_profile = enable != 0;
  g_nstages = 0;
  g_pending_stages = 0;
  return OZFP4_OK;
}

int ozfp4_stage_times(double* ms, int max, int* n_stages) {
  if (!ms || !n_stages || max < 0) return OZFP4_EINVAL;
  {
    const int rc = resolve_pending();   // asynchronous call: read its events now
    if (rc) return rc;
  }
  const int c = std::min(g_nstages, max);
  for (int i = 0; i < c; ++i) ms[i] = g_stage_ms[i];
  *n_stages = g_nstages;
  return OZFP4_OK;
}

}  // extern "C"
