// Target-model weights: layout bookkeeping, the synthetic generator and
// row-major loading into the tiled layout (gfx950).
#include <algorithm>
#include <cmath>
#include <new>

#include "model.h"

namespace sdd {

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): output for state x.
__host__ __device__ inline uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// Tensor numbering of the synthetic generator.
static int tensor_id(int kind, int layer) {
  switch (kind) {
    case SDD_T_EMBED: return 1;
    case SDD_T_LM_HEAD: return 2;
    case SDD_T_FINAL_NORM: return 3;
    default: return 16 + 16 * layer + (kind - SDD_T_WQ);
  }
}

static uint64_t tensor_key(uint64_t seed, int id) { return splitmix64(splitmix64(seed) + (uint64_t)id); }

// Irwin-Hall sum of the four 16-bit lanes of the index-th SplitMix64 output.
__device__ inline float synth_value(uint64_t key, uint64_t idx, float scale) {
  uint64_t r = splitmix64(key + idx * 0x9E3779B97F4A7C15ULL);
  int32_t s = (int32_t)(r & 0xffff) + (int32_t)((r >> 16) & 0xffff) + (int32_t)((r >> 32) & 0xffff) +
              (int32_t)(r >> 48) - 131070;
  return (float)s * scale;
}

// Source of a tiled matrix: rows of a fused matrix map to (part, logical row).
struct TiledSrc {
  int kind;  // 0 plain, 1 fused q/k/v, 2 gate/up interleaved per 16-row tile
  int K, ktile;
  MatPlan plan;   // storage order of the tiles
  int64_t N;      // physical rows
  int n0, n1;     // fused q/k/v row boundaries
  uint64_t key[3];
  const void* src[3];  // row-major sources (load); NULL parts are left untouched
  float scale;
  int gen;        // 1: synthetic values, 0: copy from src
  int bf16;
};

__device__ inline void map_row(const TiledSrc& s, int64_t row, int& part, int64_t& lrow) {
  if (s.kind == 1) {
    if (row < s.n0) { part = 0; lrow = row; }
    else if (row < s.n0 + s.n1) { part = 1; lrow = row - s.n0; }
    else { part = 2; lrow = row - s.n0 - s.n1; }
  } else if (s.kind == 2) {
    int64_t t = row / 16;
    part = (int)(t & 1);
    lrow = (t >> 1) * 16 + row % 16;
  } else {
    part = 0;
    lrow = row;
  }
}

template <typename T>
__global__ void fill_tiled_kernel(char* dst, TiledSrc s, int only_part) {
  constexpr int EPL = 16 / sizeof(T);
  const MatPlan& p = s.plan;
  const int64_t slices = plan_slots(p) * p.ng * 64;
  for (int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; id < slices;
       id += (int64_t)gridDim.x * blockDim.x) {
    // physical tile (slot, j): the j-th row tile of the unit stored at slot = i * n_wg + w, that is the i-th
    // unit of workgroup w; slots past a shorter share are padding (zero)
    const int64_t tile = id / 64;
    const int lane = (int)(id % 64);
    const int64_t slot = tile / p.ng;
    const int j = (int)(tile % p.ng);
    const uint32_t w = (uint32_t)(slot % p.n_wg), i = (uint32_t)(slot / p.n_wg);
    const uint32_t u = unit_start(w, p.KT, p.G, p.c, p.n_wg) + i;
    if (u >= unit_start(w + 1, p.KT, p.G, p.c, p.n_wg)) {
      *reinterpret_cast<uint4*>(dst + id * 16) = uint4{0, 0, 0, 0};
      continue;
    }
    const int g = (int)(u / p.KT), kt = (int)(u % p.KT);
    const int64_t nt = (int64_t)g * p.ng + j;
    const int64_t row = nt * 16 + lane % 16;
    const int k0 = kt * s.ktile + (lane / 16) * EPL;
    int part = 0;
    int64_t lrow = 0;
    if (row < s.N) map_row(s, row, part, lrow);
    if (only_part >= 0 && part != only_part) continue;
    T vals[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const int k = k0 + e;
      float v = 0.f;
      if (row < s.N && k < s.K) {
        const uint64_t idx = (uint64_t)lrow * s.K + k;
        if (s.gen) {
          v = synth_value(s.key[part], idx, s.scale);
          if (s.bf16) v = bf16_to_f32(f32_to_bf16(v));
          vals[e] = Elem<T>::from_f32(v);
          continue;
        }
        vals[e] = reinterpret_cast<const T*>(s.src[part])[idx];
        continue;
      }
      vals[e] = Elem<T>::from_f32(v);
    }
    *reinterpret_cast<uint4*>(dst + id * 16) = *reinterpret_cast<const uint4*>(vals);
  }
}

template <typename T>
__global__ void fill_rowmajor_kernel(T* dst, int64_t n, uint64_t key, float scale, const T* src) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src ? src[i] : Elem<T>::from_f32(synth_value(key, (uint64_t)i, scale));
}

__global__ void fill_f32_kernel(float* dst, int64_t n, float v, const float* src) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src ? src[i] : v;
}

static int validate_cfg(const sdd_model_config* c) {
  SDD_REQUIRE(c != nullptr, "cfg is NULL");
  SDD_REQUIRE(c->n_layers >= 0 && c->d_model > 0 && c->n_q_heads > 0 && c->n_kv_heads > 0 && c->d_ff > 0 &&
                  c->vocab > 0,
              "non-positive dimension");
  if (c->dtype != SDD_F32 && c->dtype != SDD_BF16) return fail(SDD_EUNSUPPORTED, "dtype must be SDD_F32 or SDD_BF16");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(SDD_EUNSUPPORTED, "head_dim must be 64 or 128");
  SDD_REQUIRE(c->n_q_heads % c->n_kv_heads == 0, "n_q_heads must be a multiple of n_kv_heads");
  const int ktile = c->dtype == SDD_BF16 ? 32 : 16;  // columns of one weight tile
  if (c->d_model % 32 || c->vocab % 32 || c->d_ff % ktile)
    return fail(SDD_EUNSUPPORTED, "d_model and vocab must be multiples of 32, d_ff of %d", ktile);
  SDD_REQUIRE(c->rms_eps > 0.f && c->rope_theta > 1.f, "bad rms_eps or rope_theta");
  return SDD_OK;
}

// Computes offsets; returns total bytes.
// CUs of the current device (256 when it cannot be queried): the workgroup count of the streaming plans,
// which fix the order the matrices are stored in
static int device_cus() {
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      ncu <= 0) {
    (void)hipGetLastError();
    ncu = 256;
  }
  return ncu;
}

static size_t plan_weights(const sdd_model_config* c, sdd_model* m, int n_cu) {
  const int es = c->dtype == SDD_BF16 ? 2 : 4;
  const int kt = 64 / es;  // 4 lane groups x (16 / es) elements
  const int64_t d = c->d_model, hd = c->head_dim, hq = c->n_q_heads * hd, hk = c->n_kv_heads * hd;
  // row tiles per column group
  const int ng_qkv = (int)(hd / 16);
  // o_proj has few output columns and a long K, so 128-column groups would
  // each be split over ~6 workgroups' equal shares; 64-column groups halve
  // the contributors a split group's last workgroup reduces.  (down_proj
  // streams 3x the bytes and keeps 128-column groups: their 8 KiB k-steps
  // keep more bytes in flight per wave.)
  const int ng_o = pick_ng(d / 16, false, 4);
  const int ng_gu = pick_ng(2 * (int64_t)c->d_ff / 16, true);
  const int ng_down = pick_ng(d / 16, false);
  const int ng_lm = pick_ng(c->vocab / 16, false);
  const MatPlan p_qkv = plan_matrix(hq + 2 * hk, d, kt, ng_qkv, n_cu), p_o = plan_matrix(d, hq, kt, ng_o, n_cu),
                p_gu = plan_matrix(2 * (int64_t)c->d_ff, d, kt, ng_gu, n_cu),
                p_down = plan_matrix(d, c->d_ff, kt, ng_down, n_cu), p_lm = plan_matrix(c->vocab, d, kt, ng_lm, n_cu);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  size_t e = take((size_t)c->vocab * d * es);
  size_t lm = take(plan_bytes(p_lm));
  size_t fn = take((size_t)d * 4);
  if (m) {
    m->es = es;
    m->ktile = kt;
    m->off_embed = e;
    m->off_lm = lm;
    m->off_final_norm = fn;
    m->ng_qkv = ng_qkv;
    m->ng_o = ng_o;
    m->ng_gu = ng_gu;
    m->ng_down = ng_down;
    m->ng_lm = ng_lm;
    m->plan_qkv = p_qkv;
    m->plan_o = p_o;
    m->plan_gu = p_gu;
    m->plan_down = p_down;
    m->plan_lm = p_lm;
  }
  for (int l = 0; l < c->n_layers; ++l) {
    sdd_model::Layer L;
    L.qkv = take(plan_bytes(p_qkv));
    L.o = take(plan_bytes(p_o));
    L.gu = take(plan_bytes(p_gu));
    L.down = take(plan_bytes(p_down));
    L.attn_norm = take((size_t)d * 4);
    L.ffn_norm = take((size_t)d * 4);
    L.q_norm = take((size_t)hd * 4);
    L.k_norm = take((size_t)hd * 4);
    if (m) m->layers[l] = L;
  }
  return off;
}

static int launch_blocks(int64_t work) { return (int)std::max<int64_t>(1, std::min<int64_t>(ceil_div(work, 256), 8192)); }

static int fill_tiled(sdd_model* m, char* dst, TiledSrc s, const MatPlan& plan, int only_part, hipStream_t st) {
  s.plan = plan;
  s.ktile = m->ktile;
  s.bf16 = m->cfg.dtype == SDD_BF16;
  const int64_t slices = plan_slots(plan) * plan.ng * 64;
  if (m->es == 2)
    hipLaunchKernelGGL(fill_tiled_kernel<uint16_t>, dim3(launch_blocks(slices)), dim3(256), 0, st, dst, s, only_part);
  else
    hipLaunchKernelGGL(fill_tiled_kernel<float>, dim3(launch_blocks(slices)), dim3(256), 0, st, dst, s, only_part);
  return check_launch("fill_tiled_kernel");
}

}  // namespace sdd

using namespace sdd;

extern "C" int sdd_weights_bytes(const sdd_model_config* cfg, size_t* bytes) {
  int rc = validate_cfg(cfg);
  if (rc) return rc;
  SDD_REQUIRE(bytes != nullptr, "bytes is NULL");
  *bytes = plan_weights(cfg, nullptr, device_cus());
  return SDD_OK;
}

extern "C" int sdd_model_create(const sdd_model_config* cfg, void* weights, size_t bytes, sdd_model** out) {
  int rc = validate_cfg(cfg);
  if (rc) return rc;
  SDD_REQUIRE(weights != nullptr && out != nullptr, "NULL pointer");
  SDD_REQUIRE((uintptr_t)weights % 256 == 0, "weight buffer must be 256-byte aligned");
  const int ncu = device_cus();
  size_t need = plan_weights(cfg, nullptr, ncu);
  if (bytes < need) return fail(SDD_ENOMEM, "weight buffer needs %zu bytes, got %zu", need, bytes);
  sdd_model* m = new (std::nothrow) sdd_model();
  if (!m) return fail(SDD_ENOMEM, "host allocation failed");
  m->layers = new (std::nothrow) sdd_model::Layer[std::max(1, cfg->n_layers)];
  if (!m->layers) {
    delete m;
    return fail(SDD_ENOMEM, "host allocation failed");
  }
  m->cfg = *cfg;
  m->base = reinterpret_cast<char*>(weights);
  m->bytes = bytes;
  plan_weights(cfg, m, ncu);
  m->n_cu = ncu;
  *out = m;
  return SDD_OK;
}

extern "C" int sdd_model_destroy(sdd_model* m) {
  if (m) {
    delete[] m->layers;
    delete m;
  }
  return SDD_OK;
}

extern "C" int sdd_model_init_random(sdd_model* m, uint64_t seed, float sigma, sdd_stream_t stream) {
  SDD_REQUIRE(m != nullptr, "model is NULL");
  SDD_REQUIRE(sigma >= 0.f && std::isfinite(sigma), "bad sigma");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const sdd_model_config& c = m->cfg;
  const float scale = (float)((double)sigma * 1.7320508075688772 / 65536.0);
  const int64_t d = c.d_model, hd = c.head_dim, hq = c.n_q_heads * hd, hk = c.n_kv_heads * hd;
  int rc;
  // embedding, row-major
  const int64_t ne = (int64_t)c.vocab * d;
  {
    const uint64_t key = tensor_key(seed, tensor_id(SDD_T_EMBED, 0));
    if (m->es == 2)
      hipLaunchKernelGGL(fill_rowmajor_kernel<uint16_t>, dim3(launch_blocks(ne)), dim3(256), 0, st,
                         reinterpret_cast<uint16_t*>(m->base + m->off_embed), ne, key, scale, (const uint16_t*)nullptr);
    else
      hipLaunchKernelGGL(fill_rowmajor_kernel<float>, dim3(launch_blocks(ne)), dim3(256), 0, st,
                         reinterpret_cast<float*>(m->base + m->off_embed), ne, key, scale, (const float*)nullptr);
    if ((rc = check_launch("fill_rowmajor_kernel"))) return rc;
  }
  auto gen = [&](char* dst, const MatPlan& plan, int kind, int64_t N, int K, uint64_t k0, uint64_t k1, uint64_t k2, int n0,
                 int n1) {
    TiledSrc s{};
    s.kind = kind;
    s.K = K;
    s.N = N;
    s.n0 = n0;
    s.n1 = n1;
    s.key[0] = k0;
    s.key[1] = k1;
    s.key[2] = k2;
    s.scale = scale;
    s.gen = 1;
    return fill_tiled(m, dst, s, plan, -1, st);
  };
  if ((rc = gen(m->base + m->off_lm, m->plan_lm, 0, c.vocab, (int)d, tensor_key(seed, tensor_id(SDD_T_LM_HEAD, 0)), 0, 0, 0, 0)))
    return rc;
  auto ones = [&](size_t off, int64_t n) {
    hipLaunchKernelGGL(fill_f32_kernel, dim3(launch_blocks(n)), dim3(256), 0, st,
                       reinterpret_cast<float*>(m->base + off), n, 1.0f, (const float*)nullptr);
    return check_launch("fill_f32_kernel");
  };
  if ((rc = ones(m->off_final_norm, d))) return rc;
  for (int l = 0; l < c.n_layers; ++l) {
    const sdd_model::Layer& L = m->layers[l];
    auto key = [&](int kind) { return tensor_key(seed, tensor_id(kind, l)); };
    if ((rc = gen(m->base + L.qkv, m->plan_qkv, 1, hq + 2 * hk, (int)d, key(SDD_T_WQ), key(SDD_T_WK), key(SDD_T_WV), (int)hq, (int)hk)))
      return rc;
    if ((rc = gen(m->base + L.o, m->plan_o, 0, d, (int)hq, key(SDD_T_WO), 0, 0, 0, 0))) return rc;
    if ((rc = gen(m->base + L.gu, m->plan_gu, 2, 2 * (int64_t)c.d_ff, (int)d, key(SDD_T_WGATE), key(SDD_T_WUP), 0, 0, 0))) return rc;
    if ((rc = gen(m->base + L.down, m->plan_down, 0, d, c.d_ff, key(SDD_T_WDOWN), 0, 0, 0, 0))) return rc;
    if ((rc = ones(L.attn_norm, d)) || (rc = ones(L.ffn_norm, d)) || (rc = ones(L.q_norm, hd)) || (rc = ones(L.k_norm, hd)))
      return rc;
  }
  return SDD_OK;
}

extern "C" int sdd_model_matrix_layout(const sdd_model* m, int kind, int layer, size_t* offset, size_t* bytes,
                                       int* KT, int* G, int* ng, int* n_wg, int* seg_units) {
  SDD_REQUIRE(m && offset && bytes && KT && G && ng && n_wg && seg_units, "NULL pointer");
  SDD_REQUIRE(kind == SDD_T_LM_HEAD || (kind >= SDD_T_WQ && kind <= SDD_T_WDOWN), "bad matrix kind %d", kind);
  if (kind != SDD_T_LM_HEAD) SDD_REQUIRE(layer >= 0 && layer < m->cfg.n_layers, "bad layer %d", layer);
  const MatPlan* p = nullptr;
  size_t off = 0;
  if (kind == SDD_T_LM_HEAD) {
    p = &m->plan_lm;
    off = m->off_lm;
  } else {
    const sdd_model::Layer& L = m->layers[layer];
    switch (kind) {
      case SDD_T_WQ: case SDD_T_WK: case SDD_T_WV: p = &m->plan_qkv; off = L.qkv; break;
      case SDD_T_WO: p = &m->plan_o; off = L.o; break;
      case SDD_T_WGATE: case SDD_T_WUP: p = &m->plan_gu; off = L.gu; break;
      default: p = &m->plan_down; off = L.down; break;
    }
  }
  *offset = off;
  *bytes = plan_bytes(*p);
  *KT = p->KT;
  *G = p->G;
  *ng = p->ng;
  *n_wg = p->n_wg;
  *seg_units = p->c;
  return SDD_OK;
}

extern "C" int sdd_model_load_tensor(sdd_model* m, int kind, int layer, const void* src, sdd_stream_t stream) {
  SDD_REQUIRE(m != nullptr && src != nullptr, "NULL pointer");
  SDD_REQUIRE(kind >= SDD_T_EMBED && kind <= SDD_T_K_NORM, "bad tensor kind %d", kind);
  const sdd_model_config& c = m->cfg;
  if (kind >= SDD_T_WQ) SDD_REQUIRE(layer >= 0 && layer < c.n_layers, "bad layer %d", layer);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int64_t d = c.d_model, hd = c.head_dim, hq = c.n_q_heads * hd, hk = c.n_kv_heads * hd;
  auto copy_f32 = [&](size_t off, int64_t n) {
    hipLaunchKernelGGL(fill_f32_kernel, dim3(launch_blocks(n)), dim3(256), 0, st,
                       reinterpret_cast<float*>(m->base + off), n, 0.f, reinterpret_cast<const float*>(src));
    return check_launch("fill_f32_kernel");
  };
  auto tiled = [&](size_t off, const MatPlan& plan, int skind, int64_t N, int K, int part, int n0, int n1) {
    TiledSrc s{};
    s.kind = skind;
    s.K = K;
    s.N = N;
    s.n0 = n0;
    s.n1 = n1;
    s.src[part] = src;
    s.gen = 0;
    return fill_tiled(m, m->base + off, s, plan, part, st);
  };
  if (kind == SDD_T_EMBED) {
    const int64_t ne = (int64_t)c.vocab * d;
    if (m->es == 2)
      hipLaunchKernelGGL(fill_rowmajor_kernel<uint16_t>, dim3(launch_blocks(ne)), dim3(256), 0, st,
                         reinterpret_cast<uint16_t*>(m->base + m->off_embed), ne, 0ull, 0.f,
                         reinterpret_cast<const uint16_t*>(src));
    else
      hipLaunchKernelGGL(fill_rowmajor_kernel<float>, dim3(launch_blocks(ne)), dim3(256), 0, st,
                         reinterpret_cast<float*>(m->base + m->off_embed), ne, 0ull, 0.f,
                         reinterpret_cast<const float*>(src));
    return check_launch("fill_rowmajor_kernel");
  }
  if (kind == SDD_T_LM_HEAD) return tiled(m->off_lm, m->plan_lm, 0, c.vocab, (int)d, 0, 0, 0);
  if (kind == SDD_T_FINAL_NORM) return copy_f32(m->off_final_norm, d);
  const sdd_model::Layer& L = m->layers[layer];
  switch (kind) {
    case SDD_T_WQ: return tiled(L.qkv, m->plan_qkv, 1, hq + 2 * hk, (int)d, 0, (int)hq, (int)hk);
    case SDD_T_WK: return tiled(L.qkv, m->plan_qkv, 1, hq + 2 * hk, (int)d, 1, (int)hq, (int)hk);
    case SDD_T_WV: return tiled(L.qkv, m->plan_qkv, 1, hq + 2 * hk, (int)d, 2, (int)hq, (int)hk);
    case SDD_T_WO: return tiled(L.o, m->plan_o, 0, d, (int)hq, 0, 0, 0);
    case SDD_T_WGATE: return tiled(L.gu, m->plan_gu, 2, 2 * (int64_t)c.d_ff, (int)d, 0, 0, 0);
    case SDD_T_WUP: return tiled(L.gu, m->plan_gu, 2, 2 * (int64_t)c.d_ff, (int)d, 1, 0, 0);
    case SDD_T_WDOWN: return tiled(L.down, m->plan_down, 0, d, c.d_ff, 0, 0, 0);
    case SDD_T_ATTN_NORM: return copy_f32(L.attn_norm, d);
    case SDD_T_FFN_NORM: return copy_f32(L.ffn_norm, d);
    case SDD_T_Q_NORM: return copy_f32(L.q_norm, hd);
    case SDD_T_K_NORM: return copy_f32(L.k_norm, hd);
  }
  return fail(SDD_EINVAL, "bad tensor kind %d", kind);
}
