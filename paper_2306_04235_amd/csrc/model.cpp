// model.cpp -- model-file parsing, validation, folding of the quantization
// scales into per-channel fp32 constants, and the device arena layout.
//
// Folded constants (each computed in double and rounded once to fp32):
//   int8-output linear (requantization):  scale[n] = s_in * s_w[n] / s_out,
//                                         bias[n]  = b[n] / s_out
//   fp32-output linear (dequantization):  scale[n] = s_in * s_w[n], bias = b
//   attention:  c_qk = s_q * s_k / sqrt(d_head),  c_pv = s_v / s_ctx
//   embedding:  c_emb[v] = s_E[v] * sqrt(d),  c_out[v] = s_fin * s_E[v]
//   quantization of an activation with scale s multiplies by 1 / s.
// These follow from the quantizer figure of Section 3.2: real value =
// scale * code for weights (per output channel) and activations (per tensor).
#include <cmath>
#include <cstring>
#include <string>

#include "internal.h"

namespace mnmt {
namespace {

constexpr uint32_t kI8 = 1, kF32 = 2, kI4 = 3;  // kI4: packed 4-bit weight codes

struct Entry {
  uint32_t dtype, rank, d0, d1;
  uint64_t off;
};

uint32_t rd32(const uint8_t* p) {
  uint32_t v;
  std::memcpy(&v, p, 4);
  return v;
}

// Host image of the device arena; pointers are recorded as offsets and fixed
// up once the arena address is known.
struct Image {
  std::vector<uint8_t> buf;
  std::vector<std::pair<const void**, size_t>> fix;
  size_t alloc(size_t bytes) {
    const size_t off = (buf.size() + 255) / 256 * 256;
    buf.resize(off + (bytes + 255) / 256 * 256, 0);
    return off;
  }
  template <class T>
  void bind(const T** slot, size_t off) {
    fix.push_back({reinterpret_cast<const void**>(slot), off});
  }
};

struct Parser {
  const uint8_t* blob;
  size_t n;
  std::map<std::string, Entry> t;
  std::string err;

  const Entry* get(const std::string& name, uint32_t dtype, uint32_t d0, uint32_t d1) {
    auto it = t.find(name);
    if (it == t.end()) {
      err = "missing tensor " + name;
      return nullptr;
    }
    const Entry& e = it->second;
    if (e.dtype != dtype || e.d0 != d0 || e.d1 != d1) {
      err = "tensor " + name + " has the wrong dtype or shape";
      return nullptr;
    }
    return &e;
  }
  const float* f32(const std::string& name, uint32_t d0, uint32_t d1 = 1) {
    const Entry* e = get(name, kF32, d0, d1);
    return e ? reinterpret_cast<const float*>(blob + e->off) : nullptr;
  }
  const int8_t* i8(const std::string& name, uint32_t d0, uint32_t d1) {
    const Entry* e = get(name, kI8, d0, d1);
    return e ? reinterpret_cast<const int8_t*>(blob + e->off) : nullptr;
  }
  bool positive(const std::string& name, int count, float* out) {
    const float* p = f32(name, (uint32_t)count);
    if (!p) return false;
    for (int i = 0; i < count; ++i) {
      float v;
      std::memcpy(&v, p + i, 4);
      if (!(v > 0.0f) || !std::isfinite(v)) {
        err = "scale " + name + " is not a positive finite number";
        return false;
      }
      out[i] = v;
    }
    return true;
  }
};

float rd_f(const float* p, size_t i) {
  float v;
  std::memcpy(&v, p + i, 4);
  return v;
}

// Copy an int8 weight and compute its folded constants into the image.
// 4-bit weights keep their packed rows (read by the 1-2 row decoder and the
// small-batch encoder kernels) and, unless packed_only, their int8 codes too
// (for the batched kernels).
bool add_linear(Parser& P, Image& img, LinearDev& L, const std::string& pfx, int N, int K, float s_in,
                const float* s_out, int n_blocks, bool packed_only) {
  auto it = P.t.find(pfx + ".w");
  const bool four = it != P.t.end() && it->second.dtype == kI4;
  const int8_t* w = four ? nullptr : P.i8(pfx + ".w", (uint32_t)N, (uint32_t)K);
  const uint8_t* w4 = nullptr;
  if (four) {
    if (it->second.d0 != (uint32_t)N || it->second.d1 != (uint32_t)K) {
      P.err = "tensor " + pfx + ".w has the wrong shape";
      return false;
    }
    w4 = P.blob + it->second.off;
  }
  const float* sw = P.f32(pfx + ".sw", (uint32_t)N);
  const float* b = P.f32(pfx + ".b", (uint32_t)N);
  if ((!w && !w4) || !sw || !b) return false;
  L.N = N;
  L.K = K;
  L.inv_in = (float)(1.0 / (double)s_in);
  if (four) {
    const size_t o4 = img.alloc((size_t)N * K / 2);
    std::memcpy(img.buf.data() + o4, w4, (size_t)N * K / 2);
    img.bind(&L.w4, o4);
  }
  if (!four || !packed_only) {
    const size_t ow = img.alloc((size_t)N * K);
    int8_t* dst = reinterpret_cast<int8_t*>(img.buf.data() + ow);
    if (four) {
      // in each group of 16 codes of a row, byte i (i < 8) holds code i in its
      // low nibble and code i + 8 in its high nibble, each plus 8
      for (size_t r = 0; r < (size_t)N; ++r)
        for (int g = 0; g < K / 16; ++g)
          for (int i = 0; i < 8; ++i) {
            const uint8_t byte = w4[r * (size_t)K / 2 + (size_t)g * 8 + i];
            dst[r * K + 16 * g + i] = (int8_t)((int)(byte & 15) - 8);
            dst[r * K + 16 * g + 8 + i] = (int8_t)((int)(byte >> 4) - 8);
          }
    } else {
      std::memcpy(dst, w, (size_t)N * K);
    }
    img.bind(&L.w, ow);
  }
  const size_t os = img.alloc(sizeof(float) * N), ob = img.alloc(sizeof(float) * N);
  float* sc = reinterpret_cast<float*>(img.buf.data() + os);
  float* bi = reinterpret_cast<float*>(img.buf.data() + ob);
  const int blk = N / n_blocks;
  for (int n = 0; n < N; ++n) {
    const float swn = rd_f(sw, n), bn = rd_f(b, n);
    if (!(swn > 0.0f) || !std::isfinite(swn) || !std::isfinite(bn)) {
      P.err = pfx + ": weight scale or bias not finite/positive";
      return false;
    }
    if (s_out) {
      const double so = (double)s_out[n / blk];
      sc[n] = (float)((double)s_in * (double)swn / so);
      bi[n] = (float)((double)bn / so);
    } else {
      sc[n] = (float)((double)s_in * (double)swn);
      bi[n] = bn;
    }
  }
  img.bind(&L.scale, os);
  img.bind(&L.bias, ob);
  return true;
}

bool add_ln(Parser& P, Image& img, LnDev& ln, const std::string& pfx, int d) {
  const float* g = P.f32(pfx + ".g", (uint32_t)d);
  const float* b = P.f32(pfx + ".b", (uint32_t)d);
  if (!g || !b) return false;
  const size_t og = img.alloc(sizeof(float) * d), ob = img.alloc(sizeof(float) * d);
  std::memcpy(img.buf.data() + og, g, sizeof(float) * d);
  std::memcpy(img.buf.data() + ob, b, sizeof(float) * d);
  img.bind(&ln.g, og);
  img.bind(&ln.b, ob);
  return true;
}

bool scalar(Parser& P, const std::string& name, float* v, bool positive_only) {
  const float* p = P.f32(name, 1);
  if (!p) return false;
  *v = rd_f(p, 0);
  if (!std::isfinite(*v) || (positive_only && !(*v > 0.0f))) {
    P.err = name + " is not a valid scalar";
    return false;
  }
  return true;
}

bool add_layer(Parser& P, Image& img, mnmt_model& m, LayerDev& L, const std::string& side, int l, bool dec) {
  const bool po = m.packed_only;
  const int d = m.info.d_model, F = m.info.d_ffn;
  const std::string p = side + "." + std::to_string(l);
  float s_qkv[3], s_q[1], s_kv[2], s_h[1], s_ctx, s_in;
  if (!add_ln(P, img, L.sa_ln, p + ".sa.ln", d)) return false;
  if (!P.positive(p + ".sa.qkv.sout", 3, s_qkv) || !P.positive(p + ".sa.qkv.sin", 1, &s_in)) return false;
  if (!add_linear(P, img, L.qkv, p + ".sa.qkv", 3 * d, d, s_in, s_qkv, 3, po)) return false;
  if (!P.positive(p + ".sa.o.sin", 1, &s_ctx)) return false;
  if (!add_linear(P, img, L.o, p + ".sa.o", d, d, s_ctx, nullptr, 1, po)) return false;
  L.sa_cqk = (float)((double)s_qkv[0] * (double)s_qkv[1] / std::sqrt((double)m.dh));
  L.sa_cpv = (float)((double)s_qkv[2] / (double)s_ctx);
  if (!scalar(P, p + ".sa.gamma", &L.sa_gamma, false)) return false;
  if (dec) {
    if (!add_ln(P, img, L.ca_ln, p + ".ca.ln", d)) return false;
    if (!P.positive(p + ".ca.q.sout", 1, s_q) || !P.positive(p + ".ca.q.sin", 1, &s_in)) return false;
    if (!add_linear(P, img, L.cq, p + ".ca.q", d, d, s_in, s_q, 1, po)) return false;
    if (!P.positive(p + ".ca.kv.sout", 2, s_kv)) return false;
    if (!add_linear(P, img, L.ckv, p + ".ca.kv", 2 * d, d, m.s_enc, s_kv, 2, po)) return false;
    if (!P.positive(p + ".ca.o.sin", 1, &s_ctx)) return false;
    if (!add_linear(P, img, L.co, p + ".ca.o", d, d, s_ctx, nullptr, 1, po)) return false;
    L.ca_cqk = (float)((double)s_q[0] * (double)s_kv[0] / std::sqrt((double)m.dh));
    L.ca_cpv = (float)((double)s_kv[1] / (double)s_ctx);
    if (!scalar(P, p + ".ca.gamma", &L.ca_gamma, false)) return false;
  }
  if (!add_ln(P, img, L.ff_ln, p + ".ff.ln", d)) return false;
  if (!P.positive(p + ".ff.w1.sout", 1, s_h) || !P.positive(p + ".ff.w1.sin", 1, &s_in)) return false;
  if (!add_linear(P, img, L.w1, p + ".ff.w1", F, d, s_in, s_h, 1, po)) return false;
  if (!add_linear(P, img, L.w2, p + ".ff.w2", d, F, s_h[0], nullptr, 1, po)) return false;
  return scalar(P, p + ".ff.gamma", &L.ff_gamma, false);
}

// Parse and lay out a model file; on success `img` holds the arena image and
// `m` the structure with pointers still to be fixed up.
int build_model(const void* blob, size_t n, unsigned flags, mnmt_model& m, Image*& out_img, std::string& err) {
  out_img = nullptr;
  if (flags & ~(unsigned)MNMT_LOAD_PACKED_4BIT_ONLY) {
    err = "unknown load flags";
    return MNMT_E_INVALID_ARG;
  }
  m.packed_only = (flags & MNMT_LOAD_PACKED_4BIT_ONLY) != 0;
  if (!blob || n < 64) {
    err = "model blob missing or shorter than its header";
    return MNMT_E_INVALID_ARG;
  }
  const uint8_t* p = static_cast<const uint8_t*>(blob);
  if (std::memcmp(p, "MNMT", 4) != 0 || rd32(p + 4) != 1) {
    err = "not a version-1 MNMT model file";
    return MNMT_E_BAD_MODEL;
  }
  mnmt_model_info& I = m.info;
  I.d_model = (int32_t)rd32(p + 8);
  I.n_heads = (int32_t)rd32(p + 12);
  I.d_ffn = (int32_t)rd32(p + 16);
  I.n_enc = (int32_t)rd32(p + 20);
  I.n_dec = (int32_t)rd32(p + 24);
  I.vocab = (int32_t)rd32(p + 28);
  I.max_pos = (int32_t)rd32(p + 32);
  I.ln_post = (int32_t)rd32(p + 36);
  I.pad_id = (int32_t)rd32(p + 40);
  I.bos_id = (int32_t)rd32(p + 44);
  I.eos_id = (int32_t)rd32(p + 48);
  I.unk_id = (int32_t)rd32(p + 52);
  std::memcpy(&I.ln_eps, p + 56, 4);
  const uint32_t nt = rd32(p + 60);
  if (I.d_model <= 0 || I.n_heads <= 0 || I.d_ffn <= 0 || I.n_enc < 1 || I.n_dec < 1 || I.vocab < 5 ||
      I.max_pos < 1 || (I.ln_post != 0 && I.ln_post != 1) || !(I.ln_eps > 0.0f) || !std::isfinite(I.ln_eps) ||
      nt == 0 || 64 + (uint64_t)nt * 64 > n || I.n_enc > 256 || I.n_dec > 256) {
    err = "model header has invalid dimensions";
    return MNMT_E_BAD_MODEL;
  }
  for (int id : {I.pad_id, I.bos_id, I.eos_id, I.unk_id})
    if (id < 0 || id >= I.vocab) {
      err = "special token id outside the vocabulary";
      return MNMT_E_BAD_MODEL;
    }
  if (I.d_model % I.n_heads) {
    err = "d_model is not a multiple of n_heads";
    return MNMT_E_BAD_MODEL;
  }
  m.dh = I.d_model / I.n_heads;
  if (I.d_model % 64 || I.d_ffn % 64 || I.d_model > 1024 || I.d_ffn > 8192 || m.dh % 16 || m.dh > 128) {
    err = "unsupported shape: needs d_model, d_ffn multiples of 64, d_model <= 1024, d_ffn <= 8192, "
          "head width a multiple of 16 and <= 128";
    return MNMT_E_UNSUPPORTED;
  }
  Parser P{p, n, {}, {}};
  for (uint32_t i = 0; i < nt; ++i) {
    const uint8_t* e = p + 64 + (size_t)i * 64;
    char name[41];
    std::memcpy(name, e, 40);
    name[40] = 0;
    Entry en{rd32(e + 40), rd32(e + 44), rd32(e + 48), rd32(e + 52), 0};
    std::memcpy(&en.off, e + 56, 8);
    const uint64_t bytes = en.dtype == kI4 ? (uint64_t)en.d0 * en.d1 / 2 : (uint64_t)en.d0 * en.d1 * (en.dtype == kI8 ? 1 : 4);
    if ((en.dtype != kI8 && en.dtype != kF32 && en.dtype != kI4) || (en.dtype == kI4 && en.d1 % 16) ||
        en.off % 256 || en.off + bytes > n || en.off < 64 + (uint64_t)nt * 64) {
      err = std::string("tensor ") + name + " has an invalid dtype or lies outside the file";
      return MNMT_E_BAD_MODEL;
    }
    P.t[name] = en;
  }
  auto* img = new Image();
  const int d = I.d_model, V = I.vocab, Pn = I.max_pos;
  bool ok = true;
  float s_enc = 0.f, s_fin = 0.f;
  ok = ok && scalar(P, "enc.sout", &s_enc, true) && scalar(P, "dec.sout", &s_fin, true);
  if (ok) {
    m.s_enc = s_enc;
    m.inv_enc = (float)(1.0 / (double)s_enc);
    m.inv_fin = (float)(1.0 / (double)s_fin);
    // factorized embedding (Section 2.1): E [V, Ef] and the projection P [d, Ef]
    int Ef = d;
    float s_proj = 0.f, s_u = 0.f;
    const int8_t* Pw = nullptr;
    const auto itp = P.t.find("emb.proj.w");
    if (itp != P.t.end()) {
      Ef = (int)itp->second.d1;
      Pw = P.i8("emb.proj.w", (uint32_t)d, (uint32_t)Ef);
      if (!Pw || Ef < 64 || Ef % 64 || Ef > d || !scalar(P, "emb.proj.sw", &s_proj, true) ||
          !scalar(P, "emb.proj.sout", &s_u, true)) {
        if (P.err.empty() || Pw) P.err = "factorized embedding: emb.proj.w [d, E] with E a multiple of 64 <= d, "
                                         "positive emb.proj.sw and emb.proj.sout";
        ok = false;
      }
      I.emb_dim = Ef;
      m.s_proj = s_proj;
    }
    const int8_t* E = ok ? P.i8("emb.w", (uint32_t)V, (uint32_t)Ef) : nullptr;
    const float* sE = P.f32("emb.s", (uint32_t)V);
    const float* pe = P.f32("pe", (uint32_t)Pn, (uint32_t)d);
    ok = ok && E && sE && pe;
    if (ok) {
      const size_t oE = img->alloc((size_t)V * Ef);
      std::memcpy(img->buf.data() + oE, E, (size_t)V * Ef);
      const size_t oc = img->alloc(sizeof(float) * V), oo = img->alloc(sizeof(float) * V);
      float* ce = reinterpret_cast<float*>(img->buf.data() + oc);
      float* co = reinterpret_cast<float*>(img->buf.data() + oo);
      for (int v = 0; v < V && ok; ++v) {
        const float s = rd_f(sE, v);
        if (!(s > 0.0f) || !std::isfinite(s)) {
          P.err = "embedding scale not positive";
          ok = false;
          break;
        }
        ce[v] = (float)((double)s * std::sqrt((double)d));
        co[v] = (float)((double)(Pw ? s_u : s_fin) * (double)s);
      }
      const size_t op = img->alloc(sizeof(float) * (size_t)Pn * d);
      std::memcpy(img->buf.data() + op, pe, sizeof(float) * (size_t)Pn * d);
      if (!Pw) {
        const size_t of = img->alloc(frag_bytes(V, d));  // written on the device after the upload
        img->bind(&m.E_frag, of);
      } else {
        // P [d, Ef] for the input rows; its transpose [Ef, d] with the folded
        // requantization s_fin * s_proj / s_u (no bias) for the output side
        const size_t oP = img->alloc((size_t)d * Ef), oT = img->alloc((size_t)d * Ef);
        std::memcpy(img->buf.data() + oP, Pw, (size_t)d * Ef);
        int8_t* tr = reinterpret_cast<int8_t*>(img->buf.data() + oT);
        for (int n = 0; n < d; ++n)
          for (int k = 0; k < Ef; ++k) tr[(size_t)k * d + n] = Pw[(size_t)n * Ef + k];
        const size_t os = img->alloc(sizeof(float) * Ef), ob = img->alloc(sizeof(float) * Ef);
        float* sc = reinterpret_cast<float*>(img->buf.data() + os);
        const float mu = (float)((double)s_fin * (double)s_proj / (double)s_u);
        for (int k = 0; k < Ef; ++k) sc[k] = mu;  // the bias stays zero
        img->bind(&m.proj, oP);
        img->bind(&m.proj_out.w, oT);
        img->bind(&m.proj_out.scale, os);
        img->bind(&m.proj_out.bias, ob);
        m.proj_out.N = Ef;
        m.proj_out.K = d;
        m.proj_out.inv_in = (float)(1.0 / (double)s_fin);
      }
      img->bind(&m.E, oE);
      img->bind(&m.c_emb, oc);
      img->bind(&m.c_out, oo);
      img->bind(&m.pe, op);
    }
  }
  // The layer vectors must not reallocate after bind() recorded addresses.
  m.enc.assign(I.n_enc, LayerDev{});
  m.dec.assign(I.n_dec, LayerDev{});
  m.enc_alias.assign(I.n_enc, -1);
  m.dec_alias.assign(I.n_dec, -1);
  // Cross-layer parameter sharing (Section 2.2): an int8 tensor
  // "<side>.<l>.share" = j < l makes layer l run on layer j's parameters,
  // which the arena then holds once (the copy is made after the fix-up).
  auto shared = [&](const char* side, int l, std::vector<int>& alias) {
    const std::string nm = std::string(side) + "." + std::to_string(l) + ".share";
    if (P.t.find(nm) == P.t.end()) return false;
    const int8_t* v = P.i8(nm, 1, 1);
    if (!v || v[0] < 0 || v[0] >= l) {
      if (P.err.empty() || v) P.err = nm + " must name an earlier layer";
      ok = false;
      return true;
    }
    alias[l] = v[0];
    return true;
  };
  for (int l = 0; ok && l < I.n_enc; ++l)
    if (!shared("enc", l, m.enc_alias)) ok = add_layer(P, *img, m, m.enc[l], "enc", l, false);
  for (int l = 0; ok && l < I.n_dec; ++l)
    if (!shared("dec", l, m.dec_alias)) ok = add_layer(P, *img, m, m.dec[l], "dec", l, true);
  if (ok && !I.ln_post) ok = add_ln(P, *img, m.enc_ln, "enc.ln", d) && add_ln(P, *img, m.dec_ln, "dec.ln", d);
  if (!ok) {
    err = P.err.empty() ? "model file is inconsistent" : P.err;
    delete img;
    return MNMT_E_BAD_MODEL;
  }
  if (m.packed_only) {  // every linear layer must then be 4-bit: no kernel could read the others
    bool all4 = true;
    for (auto it = P.t.begin(); it != P.t.end(); ++it) {
      const std::string& nm = it->first;
      if (nm.size() > 2 && nm.compare(nm.size() - 2, 2, ".w") == 0 && nm != "emb.w" && it->second.dtype != kI4)
        all4 = false;
    }
    if (!all4) {
      err = "MNMT_LOAD_PACKED_4BIT_ONLY needs every linear layer's weight in 4-bit";
      delete img;
      return MNMT_E_UNSUPPORTED;
    }
  }
  img->alloc(0);
  m.arena_bytes = img->buf.size();
  out_img = img;
  return MNMT_OK;
}

int finish_model(Image* img, mnmt_model& m, void* d_arena, size_t arena_bytes, hipStream_t s, std::string& err) {
  if (arena_bytes < img->buf.size()) {
    err = "model arena smaller than mnmt_model_bytes";
    return MNMT_E_INVALID_ARG;
  }
  if (reinterpret_cast<uintptr_t>(d_arena) % 256) {
    err = "model arena must be 256-byte aligned";
    return MNMT_E_INVALID_ARG;
  }
  uint8_t* base = static_cast<uint8_t*>(d_arena);
  for (auto& f : img->fix) *f.first = base + f.second;
  for (size_t l = 0; l < m.enc.size(); ++l)  // shared layers: in increasing l, so chains resolve
    if (m.enc_alias[l] >= 0) m.enc[l] = m.enc[m.enc_alias[l]];
  for (size_t l = 0; l < m.dec.size(); ++l)
    if (m.dec_alias[l] >= 0) m.dec[l] = m.dec[m.dec_alias[l]];
  hipError_t e = hipMemcpyAsync(d_arena, img->buf.data(), img->buf.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && m.E_frag)
    e = launch_pack_fragments(m.E, m.info.vocab, m.info.d_model, const_cast<int8_t*>(m.E_frag), s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    err = std::string("model upload failed: ") + hipGetErrorString(e);
    return MNMT_E_HIP;
  }
  return MNMT_OK;
}

}  // namespace

int model_size(const void* blob, size_t n, unsigned flags, size_t* bytes, std::string& err) {
  mnmt_model m;
  Image* img = nullptr;
  const int rc = build_model(blob, n, flags, m, img, err);
  if (rc == MNMT_OK) *bytes = img->buf.size();
  delete img;
  return rc;
}

int model_create(const void* blob, size_t n, unsigned flags, void* d_arena, size_t arena_bytes, hipStream_t s,
                 mnmt_model** out, std::string& err) {
  auto* m = new mnmt_model();
  Image* img = nullptr;
  int rc = build_model(blob, n, flags, *m, img, err);
  if (rc == MNMT_OK) rc = finish_model(img, *m, d_arena, arena_bytes, s, err);
  delete img;
  if (rc != MNMT_OK) {
    delete m;
    return rc;
  }
  if (hipGetDevice(&m->device) != hipSuccess) m->device = 0;
  *out = m;
  return MNMT_OK;
}

}  // namespace mnmt
