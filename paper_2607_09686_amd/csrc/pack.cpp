// Split-pack of a GGUF MoE model (no HIP dependency): the routed expert
// tensors are cut into one block per (layer, expert) and written in the
// expert-store layout the cache reads, with an index of the blocks and the
// routers in the cache's [hidden][n_experts] fp32 form.  This is the paper's
// Split-Pack Representation step: each expert tensor cut, in a fixed order,
// into one block per layer and expert, and a record per block of its kind,
// layer, expert, source offsets, byte counts, topology and a digest.
//
// GGUF (version 2 or 3): magic "GGUF", version, tensor count, metadata count,
// the metadata (key string, value type, value), the tensor infos (name, dims,
// type, offset), padding to the alignment (metadata general.alignment, default
// 32), then the tensor data; offsets are relative to the data section.  Dims
// run innermost first.  Routed experts follow the llama.cpp names per layer l:
//   blk.l.ffn_gate_exps.weight  dims (H, I, E)   rows of H inputs, per expert
//   blk.l.ffn_up_exps.weight    dims (H, I, E)
//   blk.l.ffn_down_exps.weight  dims (I, H, E)
//   blk.l.ffn_gate_inp.weight   dims (H, E)      the router, E rows of H
// so each expert's matrix is a contiguous slice of its tensor.
#include <cinttypes>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <exception>
#include <map>
#include <new>
#include <string>
#include <vector>

#include "../../include/moecache.h"

void moecache_set_last_error(const char *msg);  // moecache.cpp

namespace {

int perr(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  moecache_set_last_error(buf);
  return code;
}

enum : uint32_t { kF32 = 0, kF16 = 1, kQ4_0 = 2, kQ8_0 = 8, kQ4_K = 12, kQ6_K = 14, kBF16 = 30 };

// Bytes and weights per block of the expert block types read here (0: another type).
uint64_t block_bytes(uint32_t t, uint64_t *weights) {
  switch (t) {
    case kQ8_0: *weights = 32; return 34;
    case kQ4_0: *weights = 32; return 18;
    case kQ4_K: *weights = 256; return 144;
    case kQ6_K: *weights = 256; return 210;
    default: *weights = 0; return 0;
  }
}

// Largest hidden / intermediate width and expert count taken from a file (far above any
// model this path serves; keeps every size below 2^63).
constexpr uint64_t kMaxWidth = 1u << 16, kMaxExperts = 1u << 16;

struct Tensor {
  std::vector<uint64_t> dims;
  uint32_t type = 0;
  uint64_t offset = 0;  // absolute, in the file
};

struct Reader {
  std::FILE *f = nullptr;
  bool ok = true;
  template <class T>
  T get() {
    T v{};
    if (std::fread(&v, sizeof v, 1, f) != 1) ok = false;
    return v;
  }
  std::string str() {
    const uint64_t n = get<uint64_t>();
    if (!ok || n > (1u << 20)) {
      ok = false;
      return {};
    }
    std::string s(n, '\0');
    if (n && std::fread(&s[0], 1, n, f) != n) ok = false;
    return s;
  }
  void skip(uint64_t n) {
    if (n > (uint64_t)INT64_MAX || fseeko(f, (off_t)n, SEEK_CUR) != 0) ok = false;
  }
};

uint64_t scalar_size(uint32_t t) {
  switch (t) {
    case 0: case 1: case 7: return 1;   // uint8, int8, bool
    case 2: case 3: return 2;           // uint16, int16
    case 4: case 5: case 6: return 4;   // uint32, int32, float32
    case 10: case 11: case 12: return 8;  // uint64, int64, float64
    default: return 0;
  }
}

// One metadata value: integer values are kept (for the alignment and the expert
// counts), everything else skipped.
bool read_value(Reader &r, uint32_t type, int64_t *ival) {
  if (type == 8) {  // string
    r.str();
    return r.ok;
  }
  if (type == 9) {  // array
    const uint32_t et = r.get<uint32_t>();
    const uint64_t n = r.get<uint64_t>();
    if (!r.ok) return false;
    if (et == 8) {
      for (uint64_t i = 0; i < n && r.ok; ++i) r.str();
    } else if (et == 9 || scalar_size(et) == 0) {
      return false;  // nested arrays are not used by the models this reads
    } else {
      uint64_t bytes = 0;
      if (__builtin_mul_overflow(n, scalar_size(et), &bytes)) return false;
      r.skip(bytes);
    }
    return r.ok;
  }
  const uint64_t sz = scalar_size(type);
  if (!sz) return false;
  uint64_t v = 0;
  if (std::fread(&v, sz, 1, r.f) != 1) return false;
  if (ival) {
    if (type == 1) *ival = (int8_t)v;
    else if (type == 3) *ival = (int16_t)v;
    else if (type == 5) *ival = (int32_t)v;
    else if (type == 6 || type == 12) *ival = -1;  // floating point: not an integer setting
    else *ival = (int64_t)v;
  }
  return true;
}

// FNV-1a, 64 bits, of a byte range (continuing from h).
uint64_t fnv1a(const uint8_t *p, size_t n, uint64_t h = 0xcbf29ce484222325ull) {
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 0x100000001b3ull;
  }
  return h;
}

float half_to_float(uint16_t h) {
  const uint32_t s = (uint32_t)(h >> 15) << 31, e = (h >> 10) & 0x1f, m = h & 0x3ff;
  uint32_t bits;
  if (e == 0) {
    if (m == 0) {
      bits = s;
    } else {  // subnormal: m * 2^-24
      float v = (float)m * (1.0f / 16777216.0f);
      std::memcpy(&bits, &v, 4);
      bits |= s;
    }
  } else if (e == 31) {
    bits = s | 0x7f800000u | (m << 13);
  } else {
    bits = s | ((e + 112) << 23) | (m << 13);
  }
  float f;
  std::memcpy(&f, &bits, 4);
  return f;
}

bool read_at(std::FILE *f, uint64_t off, void *dst, size_t n) {
  return off <= (uint64_t)INT64_MAX && fseeko(f, (off_t)off, SEEK_SET) == 0 &&
         std::fread(dst, 1, n, f) == n;
}

struct Closer {
  std::FILE *f;
  ~Closer() {
    if (f) std::fclose(f);
  }
};

int pack_gguf(const char *gguf_path, const char *pack_path, const char *index_path,
              const char *router_path, moe_pack_info *info) {
  std::memset(info, 0, sizeof *info);
  Reader r;
  r.f = std::fopen(gguf_path, "rb");
  if (!r.f) return perr(MOE_EIO, "cannot open %s", gguf_path);
  Closer cin{r.f};
  const uint32_t magic = r.get<uint32_t>(), version = r.get<uint32_t>();
  if (!r.ok || magic != 0x46554747u) return perr(MOE_EINVAL, "%s is not a GGUF file", gguf_path);
  if (version < 2 || version > 3) return perr(MOE_EINVAL, "GGUF version %u is not read", version);
  const uint64_t n_tensors = r.get<uint64_t>(), n_kv = r.get<uint64_t>();
  if (!r.ok || n_tensors > (1u << 24) || n_kv > (1u << 24)) return perr(MOE_EINVAL, "bad GGUF header");
  int64_t alignment = 32, used = 0;
  for (uint64_t i = 0; i < n_kv; ++i) {
    const std::string key = r.str();
    const uint32_t type = r.get<uint32_t>();
    if (!r.ok) return perr(MOE_EINVAL, "truncated GGUF metadata");
    int64_t v = -1;
    if (!read_value(r, type, &v)) return perr(MOE_EINVAL, "bad GGUF metadata value for %s", key.c_str());
    if (key == "general.alignment" && v > 0) alignment = v;
    const std::string suffix = ".expert_used_count";
    if (key.size() > suffix.size() && key.compare(key.size() - suffix.size(), suffix.size(), suffix) == 0 &&
        v > 0 && v <= (int64_t)kMaxExperts)
      used = v;
  }
  std::map<std::string, Tensor> tensors;
  for (uint64_t i = 0; i < n_tensors; ++i) {
    Tensor t;
    const std::string name = r.str();
    const uint32_t nd = r.get<uint32_t>();
    if (!r.ok || nd > 8) return perr(MOE_EINVAL, "bad GGUF tensor info");
    for (uint32_t d = 0; d < nd; ++d) t.dims.push_back(r.get<uint64_t>());
    t.type = r.get<uint32_t>();
    t.offset = r.get<uint64_t>();
    if (!r.ok) return perr(MOE_EINVAL, "truncated GGUF tensor info");
    tensors[name] = t;
  }
  const off_t pos = ftello(r.f);
  if (pos < 0 || alignment <= 0 || alignment > (1 << 20) || (alignment & (alignment - 1)))
    return perr(MOE_EINVAL, "bad GGUF alignment %" PRId64, alignment);
  if (fseeko(r.f, 0, SEEK_END) != 0) return perr(MOE_EIO, "cannot seek in %s", gguf_path);
  const off_t fend = ftello(r.f);
  if (fend < pos) return perr(MOE_EIO, "cannot size %s", gguf_path);
  const uint64_t file_bytes = (uint64_t)fend;
  const uint64_t data0 = ((uint64_t)pos + alignment - 1) / alignment * alignment;
  for (auto &kv : tensors) {
    if (kv.second.offset > file_bytes) return perr(MOE_EINVAL, "tensor %s starts past the end of the file",
                                                  kv.first.c_str());
    kv.second.offset += data0;
  }

  // the routed-expert layers: consecutive from 0
  int32_t L = 0;
  auto name = [](int l, const char *what) { return "blk." + std::to_string(l) + "." + what + ".weight"; };
  while (tensors.count(name(L, "ffn_gate_exps"))) ++L;
  if (L == 0) return perr(MOE_EINVAL, "no routed expert tensors (blk.0.ffn_gate_exps.weight)");
  const Tensor &g0 = tensors[name(0, "ffn_gate_exps")];
  if (g0.dims.size() != 3) return perr(MOE_EINVAL, "expert tensors must have 3 dims");
  const uint64_t H = g0.dims[0], I = g0.dims[1], E = g0.dims[2];
  // gate and up share one block type, down may have another (the Q4_K_M mix); each is the
  // same in every layer, so that every slot holds P bytes
  const uint32_t qt = g0.type;
  uint64_t wgu = 0, wdn = 0;
  const uint64_t bgu = block_bytes(qt, &wgu);
  if (!bgu)
    return perr(MOE_EINVAL, "expert tensors of ggml type %u: only Q8_0 (8), Q4_0 (2), Q4_K (12) and "
                "Q6_K (14) are read", qt);
  auto d0 = tensors.find(name(0, "ffn_down_exps"));
  if (d0 == tensors.end()) return perr(MOE_EINVAL, "missing %s", name(0, "ffn_down_exps").c_str());
  const uint32_t qd = d0->second.type;
  const uint64_t bdn = block_bytes(qd, &wdn);
  if (!bdn)
    return perr(MOE_EINVAL, "down expert tensors of ggml type %u: only Q8_0 (8), Q4_0 (2), Q4_K (12) "
                "and Q6_K (14) are read", qd);
  if (H == 0 || I == 0 || H > kMaxWidth || I > kMaxWidth || H % wgu || I % wdn || E < 1 || E > kMaxExperts)
    return perr(MOE_EINVAL, "bad expert shape (hidden %" PRIu64 ", inter %" PRIu64 ", experts %" PRIu64 ")",
                H, I, E);
  // sizes below 2^16 * 2^16 * 2 bytes per matrix, 2^34 * 3 per payload: no overflow
  const uint64_t M = I * (H / wgu) * bgu, Md = H * (I / wdn) * bdn, P = 2 * M + Md;
  uint64_t pack_total = 0;
  if (__builtin_mul_overflow(P, E * (uint64_t)L, &pack_total))
    return perr(MOE_EINVAL, "the pack would exceed 2^64 bytes");
  for (int32_t l = 0; l < L; ++l) {
    const char *kinds[3] = {"ffn_gate_exps", "ffn_up_exps", "ffn_down_exps"};
    for (int m = 0; m < 3; ++m) {
      auto it = tensors.find(name(l, kinds[m]));
      if (it == tensors.end()) return perr(MOE_EINVAL, "missing %s", name(l, kinds[m]).c_str());
      const Tensor &t = it->second;
      const bool ok = t.dims.size() == 3 && t.type == (m < 2 ? qt : qd) && t.dims[2] == E &&
                      (m < 2 ? (t.dims[0] == H && t.dims[1] == I) : (t.dims[0] == I && t.dims[1] == H));
      if (!ok)
        return perr(MOE_EINVAL, "%s does not match blk.0's experts (shape, or a block type that "
                    "differs between layers)", name(l, kinds[m]).c_str());
      const uint64_t bytes = E * (m < 2 ? M : Md);  // <= 2^16 * 2^34
      if (t.offset > file_bytes || bytes > file_bytes - t.offset)
        return perr(MOE_EINVAL, "%s runs past the end of the file", name(l, kinds[m]).c_str());
    }
    if (router_path) {
      auto it = tensors.find(name(l, "ffn_gate_inp"));
      if (it == tensors.end() || it->second.dims.size() != 2 || it->second.dims[0] != H ||
          it->second.dims[1] != E ||
          (it->second.type != kF32 && it->second.type != kF16 && it->second.type != kBF16))
        return perr(MOE_EINVAL, "router %s missing or not an F32 / F16 / BF16 (H, E) tensor",
                    name(l, "ffn_gate_inp").c_str());
      const uint64_t rbytes = H * E * (it->second.type == kF32 ? 4 : 2);
      if (it->second.offset > file_bytes || rbytes > file_bytes - it->second.offset)
        return perr(MOE_EINVAL, "router %s runs past the end of the file", name(l, "ffn_gate_inp").c_str());
    }
  }

  std::FILE *fp = std::fopen(pack_path, "wb");
  if (!fp) return perr(MOE_EIO, "cannot create %s", pack_path);
  Closer cp{fp};
  std::FILE *fi = std::fopen(index_path, "w");
  if (!fi) return perr(MOE_EIO, "cannot create %s", index_path);
  Closer ci{fi};
  std::string src_json;  // the source path as a JSON string body
  for (const char *q = gguf_path; *q; ++q) {
    if (*q == '"' || *q == '\\') src_json += '\\';
    if ((unsigned char)*q >= 0x20) src_json += *q;
  }
  std::fprintf(fi, "{\"format\": \"moecache expert pack\", \"source\": \"%s\", \"n_layers\": %d, "
               "\"n_experts\": %" PRIu64 ", \"top_k\": %" PRId64 ", \"hidden\": %" PRIu64
               ", \"inter\": %" PRIu64 ", \"qtype\": %u, \"payload_bytes\": %" PRIu64 "}\n",
               src_json.c_str(), L, E, used, H, I, qt == qd ? qt : qt | (qd << 8), P);
  std::vector<uint8_t> buf(P);
  uint64_t out = 0, digest_all = 0xcbf29ce484222325ull;
  for (int32_t l = 0; l < L; ++l) {
    const Tensor &tg = tensors[name(l, "ffn_gate_exps")], &tu = tensors[name(l, "ffn_up_exps")],
                 &td = tensors[name(l, "ffn_down_exps")];
    for (uint64_t e = 0; e < E; ++e) {
      const uint64_t src[3] = {tg.offset + e * M, tu.offset + e * M, td.offset + e * Md};
      const uint64_t len[3] = {M, M, Md};
      for (int m = 0; m < 3; ++m)
        if (!read_at(r.f, src[m], buf.data() + m * M, len[m]))
          return perr(MOE_EIO, "short read in %s (layer %d expert %" PRIu64 ")", gguf_path, l, e);
      if (std::fwrite(buf.data(), 1, P, fp) != P) return perr(MOE_EIO, "short write to %s", pack_path);
      const uint64_t dg = fnv1a(buf.data(), P);
      digest_all = fnv1a(reinterpret_cast<const uint8_t *>(&dg), 8, digest_all);
      std::fprintf(fi, "{\"layer\": %d, \"expert\": %" PRIu64 ", \"offset\": %" PRIu64 ", \"bytes\": %" PRIu64
                   ", \"gate\": [%" PRIu64 ", %" PRIu64 "], \"up\": [%" PRIu64 ", %" PRIu64
                   "], \"down\": [%" PRIu64 ", %" PRIu64 "], \"fnv1a64\": \"%016" PRIx64 "\"}\n",
                   l, e, out, P, src[0], M, src[1], M, src[2], Md, dg);
      out += P;
    }
  }
  if (router_path) {
    std::FILE *fr = std::fopen(router_path, "wb");
    if (!fr) return perr(MOE_EIO, "cannot create %s", router_path);
    Closer cr{fr};
    std::vector<float> wr(H * E);
    for (int32_t l = 0; l < L; ++l) {
      const Tensor &t = tensors[name(l, "ffn_gate_inp")];
      const uint64_t es = t.type == kF32 ? 4 : 2;
      std::vector<uint8_t> raw(H * E * es);
      if (!read_at(r.f, t.offset, raw.data(), raw.size()))
        return perr(MOE_EIO, "short read of the router of layer %d", l);
      // GGUF holds E rows of H; the cache takes [H][E]
      for (uint64_t e = 0; e < E; ++e)
        for (uint64_t h = 0; h < H; ++h) {
          const uint64_t i = e * H + h;
          float v;
          if (t.type == kF32) {
            std::memcpy(&v, raw.data() + 4 * i, 4);
          } else {
            uint16_t b;
            std::memcpy(&b, raw.data() + 2 * i, 2);
            if (t.type == kF16) {
              v = half_to_float(b);
            } else {
              const uint32_t bits = (uint32_t)b << 16;
              std::memcpy(&v, &bits, 4);
            }
          }
          wr[h * E + e] = v;
        }
      if (std::fwrite(wr.data(), 4, wr.size(), fr) != wr.size())
        return perr(MOE_EIO, "short write to %s", router_path);
    }
  }
  std::fprintf(fi, "{\"blocks\": %" PRIu64 ", \"pack_bytes\": %" PRIu64 ", \"fnv1a64_of_digests\": \"%016" PRIx64
               "\"}\n", (uint64_t)L * E, out, digest_all);
  info->n_layers = L;
  info->n_experts = (int32_t)E;
  info->top_k = (int32_t)used;
  info->hidden = (int32_t)H;
  info->inter = (int32_t)I;
  info->qtype = (int32_t)(qt == qd ? qt : qt | (qd << 8));
  info->payload_bytes = P;
  info->pack_bytes = out;
  return MOE_OK;
}

}  // namespace

extern "C" int moe_pack_gguf(const char *gguf_path, const char *pack_path, const char *index_path,
                             const char *router_path, moe_pack_info *info) {
  if (!gguf_path || !pack_path || !index_path || !info)
    return perr(MOE_EINVAL, "moe_pack_gguf: NULL argument");
  try {
    return pack_gguf(gguf_path, pack_path, index_path, router_path, info);
  } catch (const std::bad_alloc &) {
    return perr(MOE_ENOMEM, "moe_pack_gguf: out of host memory");
  } catch (const std::exception &ex) {
    return perr(MOE_EINVAL, "moe_pack_gguf: %s", ex.what());
  }
}
