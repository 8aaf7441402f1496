// gockpt_persist.cpp -- persistence of a restored checkpoint (Sec. 4.4.3) and
// its reading back for a restart (Sec. 4.3.2).  Host only.
//
// A checkpoint is a directory:
//   data.bin  master | exp_avg | exp_avg_sq, fp32[n] each, every array at a
//             4 KiB-aligned offset;
//   user      optional caller text (step counters, throughput history, ...);
//   meta      the scalar state, the hyperparameters, the layout and a CRC-32C
//             of every piece of data.bin -- written last, to meta.tmp, synced
//             and renamed, so a checkpoint is complete exactly when `meta`
//             exists (the paper writes its metadata after the tensors to mark
//             the checkpoint usable).
// Several threads write (and read) data.bin in pieces at their own offsets
// (Sec. 4.4.1 uses parallel writers to fill the SSD's bandwidth).
#include <dirent.h>
#include <errno.h>
#include <fcntl.h>
#include <nmmintrin.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <sys/stat.h>
#include <unistd.h>

#include <atomic>
#include <chrono>
#include <string>
#include <thread>
#include <vector>

#include "../../include/gockpt.h"

namespace gockpt {
void set_host_error(const std::string& msg);
}

namespace {

constexpr uint64_t kAlign = 4096;
constexpr const char* kMagic = "gockpt-checkpoint 1";

uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// CRC-32C (Castagnoli) with the SSE4.2 instruction, 8 bytes at a time.
uint32_t crc32c(const uint8_t* p, uint64_t len) {
    uint64_t c = 0xFFFFFFFFu;
    while (len >= 8) {
        uint64_t v;
        memcpy(&v, p, 8);
        c = _mm_crc32_u64(c, v);
        p += 8;
        len -= 8;
    }
    uint32_t c32 = static_cast<uint32_t>(c);
    while (len--) c32 = _mm_crc32_u8(c32, *p++);
    return c32 ^ 0xFFFFFFFFu;
}

struct Piece {
    int array;        // 0 master, 1 exp_avg, 2 exp_avg_sq
    uint64_t offset;  // byte offset inside the array
    uint64_t bytes;
};

struct Layout {
    uint64_t array_bytes, stride, total, piece;
    std::vector<Piece> pieces;
    std::vector<size_t> first;  // index of each array's first piece
};

Layout make_layout(int64_t n, uint64_t piece) {
    Layout L;
    L.array_bytes = 4ull * static_cast<uint64_t>(n);
    L.stride = round_up(L.array_bytes, kAlign);
    L.total = 2 * L.stride + L.array_bytes;
    L.piece = piece;
    for (int a = 0; a < 3; ++a) {
        L.first.push_back(L.pieces.size());
        for (uint64_t o = 0; o < L.array_bytes; o += piece)
            L.pieces.push_back({a, o, L.array_bytes - o < piece ? L.array_bytes - o : piece});
    }
    L.first.push_back(L.pieces.size());
    return L;
}

int fail(int code, const std::string& msg) {
    gockpt::set_host_error(msg);
    return code;
}

std::string path_join(const char* dir, const char* name) {
    std::string p(dir);
    if (!p.empty() && p.back() != '/') p += '/';
    return p + name;
}

bool write_all(int fd, const void* buf, size_t len) {
    const uint8_t* p = static_cast<const uint8_t*>(buf);
    while (len > 0) {
        const ssize_t w = write(fd, p, len);
        if (w < 0) {
            if (errno == EINTR) continue;
            return false;
        }
        p += w;
        len -= static_cast<size_t>(w);
    }
    return true;
}

bool pwrite_all(int fd, const uint8_t* p, uint64_t len, uint64_t off) {
    while (len > 0) {
        const ssize_t w = pwrite(fd, p, len, static_cast<off_t>(off));
        if (w < 0) {
            if (errno == EINTR) continue;
            return false;
        }
        p += w;
        off += static_cast<uint64_t>(w);
        len -= static_cast<uint64_t>(w);
    }
    return true;
}

bool pread_all(int fd, uint8_t* p, uint64_t len, uint64_t off) {
    while (len > 0) {
        const ssize_t r = pread(fd, p, len, static_cast<off_t>(off));
        if (r < 0) {
            if (errno == EINTR) continue;
            return false;
        }
        if (r == 0) {  // short file: no errno of its own
            errno = 0;
            return false;
        }
        p += r;
        off += static_cast<uint64_t>(r);
        len -= static_cast<uint64_t>(r);
    }
    return true;
}

bool sync_dir(const char* dir) {
    const int fd = open(dir, O_RDONLY | O_DIRECTORY);
    if (fd < 0) return false;
    const bool ok = fsync(fd) == 0;
    close(fd);
    return ok;
}

// The files a checkpoint directory holds.
const char* const kCkptFiles[] = {"meta", "meta.tmp", "user", "data.bin"};

// Remove a checkpoint directory this library wrote (its own files only; a
// directory that holds anything else is left in place).  Missing is fine.
void remove_ckpt_dir(const std::string& d) {
    for (const char* f : kCkptFiles) (void)unlink(path_join(d.c_str(), f).c_str());
    (void)rmdir(d.c_str());
}

std::string parent_of(const std::string& d) {
    const size_t k = d.find_last_of('/');
    if (k == std::string::npos) return ".";
    return k == 0 ? "/" : d.substr(0, k);
}

// Put the complete checkpoint directory `tmp` at `d`.  Where d already holds
// a checkpoint the two are exchanged in one step (renameat2 RENAME_EXCHANGE),
// so d holds a complete checkpoint at every moment; the old one is then
// removed.  On a file system without the exchange, d is first moved aside.
bool install_dir(const std::string& tmp, const std::string& d, std::string& err) {
    struct stat st;
    if (stat(d.c_str(), &st) != 0) {
        if (errno != ENOENT) return (err = std::string("stat ") + d + ": " + strerror(errno)), false;
        if (rename(tmp.c_str(), d.c_str()) != 0) return (err = std::string("rename: ") + strerror(errno)), false;
    } else if (renameat2(AT_FDCWD, tmp.c_str(), AT_FDCWD, d.c_str(), RENAME_EXCHANGE) == 0) {
        remove_ckpt_dir(tmp);  // now the old checkpoint
    } else {
        if (errno != EINVAL && errno != ENOSYS && errno != EOPNOTSUPP)
            return (err = std::string("renameat2: ") + strerror(errno)), false;
        const std::string old = d + ".gockpt-old";
        remove_ckpt_dir(old);
        if (rename(d.c_str(), old.c_str()) != 0 || rename(tmp.c_str(), d.c_str()) != 0)
            return (err = std::string("rename: ") + strerror(errno)), false;
        remove_ckpt_dir(old);
    }
    if (!sync_dir(parent_of(d).c_str())) return (err = "sync parent directory"), false;
    return true;
}

// Run body(piece_index) over all pieces with nthreads workers.
template <class F>
bool parallel_pieces(size_t count, int nthreads, F body) {
    std::atomic<size_t> next{0};
    std::atomic<bool> ok{true};
    auto worker = [&]() {
        for (;;) {
            const size_t k = next.fetch_add(1);
            if (k >= count || !ok.load()) return;
            if (!body(k)) ok = false;
        }
    };
    if (nthreads <= 0) nthreads = 16;
    if (static_cast<size_t>(nthreads) > count) nthreads = count ? static_cast<int>(count) : 1;
    std::vector<std::thread> pool;
    for (int i = 1; i < nthreads; ++i) pool.emplace_back(worker);
    worker();
    for (auto& t : pool) t.join();
    return ok.load();
}

std::string hexf(double x) {
    char b[64];
    snprintf(b, sizeof b, "%a", x);
    return b;
}

struct Meta {
    int64_t n = -1, t = 0, tracker = 0;
    double scale = 1.0;
    int32_t K = 0, skipped = 0;
    double beta1 = 0, beta2 = 0, eps = 0, wd = 0;
    uint64_t piece = 0, stride = 0, array_bytes = 0, total = 0;
    std::vector<uint32_t> crc[3];
    bool has_user = false;
};

bool parse_meta(const std::string& text, Meta* m, std::string& err) {
    size_t pos = 0;
    bool magic = false;
    while (pos < text.size()) {
        size_t e = text.find('\n', pos);
        if (e == std::string::npos) e = text.size();
        const std::string line = text.substr(pos, e - pos);
        pos = e + 1;
        if (line.empty()) continue;
        if (line == kMagic) {
            magic = true;
            continue;
        }
        const size_t sp = line.find(' ');
        if (sp == std::string::npos) {
            err = "meta: malformed line";
            return false;
        }
        const std::string k = line.substr(0, sp), v = line.substr(sp + 1);
        const char* s = v.c_str();
        if (k == "n") m->n = strtoll(s, nullptr, 10);
        else if (k == "t") m->t = strtoll(s, nullptr, 10);
        else if (k == "tracker") m->tracker = strtoll(s, nullptr, 10);
        else if (k == "scale") m->scale = strtod(s, nullptr);
        else if (k == "K") m->K = static_cast<int32_t>(strtol(s, nullptr, 10));
        else if (k == "skipped") m->skipped = static_cast<int32_t>(strtol(s, nullptr, 10));
        else if (k == "beta1") m->beta1 = strtod(s, nullptr);
        else if (k == "beta2") m->beta2 = strtod(s, nullptr);
        else if (k == "eps") m->eps = strtod(s, nullptr);
        else if (k == "weight_decay") m->wd = strtod(s, nullptr);
        else if (k == "piece_bytes") m->piece = strtoull(s, nullptr, 10);
        else if (k == "array_stride") m->stride = strtoull(s, nullptr, 10);
        else if (k == "array_bytes") m->array_bytes = strtoull(s, nullptr, 10);
        else if (k == "data_bytes") m->total = strtoull(s, nullptr, 10);
        else if (k == "user") m->has_user = v == "1";
        else if (k == "crc_master" || k == "crc_exp_avg" || k == "crc_exp_avg_sq") {
            const int a = k == "crc_master" ? 0 : (k == "crc_exp_avg" ? 1 : 2);
            const char* q = s;
            while (*q) {
                char* end = nullptr;
                const unsigned long x = strtoul(q, &end, 16);
                if (end == q) break;
                m->crc[a].push_back(static_cast<uint32_t>(x));
                q = *end == ',' ? end + 1 : end;
            }
        }
    }
    if (!magic) {
        err = "meta: not a gockpt checkpoint";
        return false;
    }
    if (m->n < 0 || m->piece == 0 || m->piece % kAlign != 0) {
        err = "meta: missing n or piece size";
        return false;
    }
    return true;
}

bool read_file(const std::string& path, std::string* out) {
    FILE* f = fopen(path.c_str(), "rb");
    if (f == nullptr) return false;
    char buf[65536];
    size_t r;
    out->clear();
    while ((r = fread(buf, 1, sizeof buf, f)) > 0) out->append(buf, r);
    const bool ok = !ferror(f);
    fclose(f);
    return ok;
}

void to_info(const Meta& m, gockpt_ckpt_info* info) {
    memset(info, 0, sizeof *info);
    info->n = m.n;
    info->t = m.t;
    info->tracker = m.tracker;
    info->scale = static_cast<float>(m.scale);
    info->K = m.K;
    info->skipped = m.skipped;
    info->beta1 = m.beta1;
    info->beta2 = m.beta2;
    info->eps = m.eps;
    info->weight_decay = m.wd;
    info->piece_bytes = m.piece;
    info->data_bytes = m.total;
    info->has_user = m.has_user ? 1 : 0;
}

int load_meta(const char* dir, Meta* m) {
    if (dir == nullptr) return fail(GOCKPT_EINVAL, "checkpoint directory is NULL");
    std::string text;
    if (!read_file(path_join(dir, "meta"), &text))
        return fail(GOCKPT_EFAILED, std::string("no complete checkpoint in ") + dir + " (meta missing)");
    std::string err;
    if (!parse_meta(text, m, err)) return fail(GOCKPT_EFAILED, err);
    const Layout L = make_layout(m->n, m->piece);
    if (m->stride != L.stride || m->array_bytes != L.array_bytes || m->total != L.total)
        return fail(GOCKPT_EFAILED, "meta: layout does not match n");
    for (int a = 0; a < 3; ++a)
        if (m->crc[a].size() != L.first[a + 1] - L.first[a]) return fail(GOCKPT_EFAILED, "meta: checksum count");
    return GOCKPT_OK;
}

}  // namespace

extern "C" {

int gockpt_write_checkpoint(const char* dir, const float* master, const float* exp_avg, const float* exp_avg_sq,
                            const gockpt_ckpt_info* info, const char* user_meta, int nthreads,
                            gockpt_io_stats* stats) {
    const auto t0 = std::chrono::steady_clock::now();
    if (dir == nullptr || info == nullptr || info->n < 0) return fail(GOCKPT_EINVAL, "write_checkpoint: bad arguments");
    if (info->n > 0 && (master == nullptr || exp_avg == nullptr || exp_avg_sq == nullptr))
        return fail(GOCKPT_EINVAL, "write_checkpoint: NULL array");
    const uint64_t piece = info->piece_bytes ? info->piece_bytes : (64ull << 20);
    if (piece % kAlign != 0) return fail(GOCKPT_EINVAL, "write_checkpoint: piece_bytes must be a multiple of 4096");
    // The checkpoint is written into a sibling directory and put in place
    // last, so a directory that already holds a complete checkpoint keeps it
    // until the new one is complete (a crash while writing loses nothing).
    std::string target(dir);
    while (target.size() > 1 && target.back() == '/') target.pop_back();
    const std::string work = target + ".gockpt-tmp";
    remove_ckpt_dir(work);  // left over from an interrupted write
    if (mkdir(work.c_str(), 0755) != 0)
        return fail(GOCKPT_EFAILED, std::string("write_checkpoint: mkdir ") + work + ": " + strerror(errno));
    const std::string meta_path = path_join(work.c_str(), "meta"), tmp_path = path_join(work.c_str(), "meta.tmp");

    const Layout L = make_layout(info->n, piece);
    const std::string data_path = path_join(work.c_str(), "data.bin");
    const int fd = open(data_path.c_str(), O_CREAT | O_WRONLY | O_TRUNC, 0644);
    // every failure from here on removes the half-written sibling directory
    auto bail = [&](const std::string& msg) {
        remove_ckpt_dir(work);
        return fail(GOCKPT_EFAILED, msg);
    };
    if (fd < 0) return bail(std::string("write_checkpoint: open data.bin: ") + strerror(errno));
    if (ftruncate(fd, static_cast<off_t>(L.total)) != 0) {
        const int e = errno;
        close(fd);
        return bail(std::string("write_checkpoint: ftruncate: ") + strerror(e));
    }
    const uint8_t* src[3] = {reinterpret_cast<const uint8_t*>(master), reinterpret_cast<const uint8_t*>(exp_avg),
                             reinterpret_cast<const uint8_t*>(exp_avg_sq)};
    std::vector<uint32_t> crc(L.pieces.size());
    std::atomic<int> io_errno{0};  // errno is per thread: keep the writer's
    const bool ok = parallel_pieces(L.pieces.size(), nthreads, [&](size_t k) {
        const Piece& p = L.pieces[k];
        const uint8_t* s = src[p.array] + p.offset;
        crc[k] = crc32c(s, p.bytes);
        if (pwrite_all(fd, s, p.bytes, p.array * L.stride + p.offset)) return true;
        io_errno = errno;
        return false;
    });
    const bool synced = ok && fdatasync(fd) == 0;
    if (ok && !synced) io_errno = errno;
    close(fd);
    if (!ok || !synced)
        return bail(std::string("write_checkpoint: writing data.bin: ") + strerror(io_errno.load()));
    const bool user = user_meta != nullptr;
    if (user) {
        const std::string up = path_join(work.c_str(), "user");
        const int ufd = open(up.c_str(), O_CREAT | O_WRONLY | O_TRUNC, 0644);
        const bool uok = ufd >= 0 && write_all(ufd, user_meta, strlen(user_meta)) && fsync(ufd) == 0;
        if (ufd >= 0) close(ufd);
        if (!uok) return bail("write_checkpoint: writing user");
    }
    std::string m = std::string(kMagic) + "\n";
    m += "n " + std::to_string(info->n) + "\n";
    m += "t " + std::to_string(info->t) + "\n";
    m += "tracker " + std::to_string(info->tracker) + "\n";
    m += "scale " + hexf(info->scale) + "\n";
    m += "K " + std::to_string(info->K) + "\n";
    m += "skipped " + std::to_string(info->skipped) + "\n";
    m += "beta1 " + hexf(info->beta1) + "\n";
    m += "beta2 " + hexf(info->beta2) + "\n";
    m += "eps " + hexf(info->eps) + "\n";
    m += "weight_decay " + hexf(info->weight_decay) + "\n";
    m += "piece_bytes " + std::to_string(piece) + "\n";
    m += "array_stride " + std::to_string(L.stride) + "\n";
    m += "array_bytes " + std::to_string(L.array_bytes) + "\n";
    m += "data_bytes " + std::to_string(L.total) + "\n";
    m += std::string("user ") + (user ? "1" : "0") + "\n";
    const char* names[3] = {"crc_master", "crc_exp_avg", "crc_exp_avg_sq"};
    for (int a = 0; a < 3; ++a) {
        m += names[a];
        m += ' ';
        char b[16];
        for (size_t k = L.first[a]; k < L.first[a + 1]; ++k) {
            snprintf(b, sizeof b, k + 1 < L.first[a + 1] ? "%08x," : "%08x", crc[k]);
            m += b;
        }
        m += '\n';
    }
    const int mfd = open(tmp_path.c_str(), O_CREAT | O_WRONLY | O_TRUNC, 0644);
    const bool mok = mfd >= 0 && write_all(mfd, m.data(), m.size()) && fsync(mfd) == 0;
    if (mfd >= 0) close(mfd);
    if (!mok) return bail("write_checkpoint: writing meta.tmp");
    if (rename(tmp_path.c_str(), meta_path.c_str()) != 0 || !sync_dir(work.c_str()))
        return bail(std::string("write_checkpoint: committing meta: ") + strerror(errno));
    std::string ierr;
    if (!install_dir(work, target, ierr)) return bail("write_checkpoint: " + ierr);
    if (stats != nullptr) {
        stats->bytes = static_cast<double>(3 * L.array_bytes);
        stats->ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
        stats->pieces = static_cast<int64_t>(L.pieces.size());
    }
    return GOCKPT_OK;
}

int gockpt_read_checkpoint_info(const char* dir, gockpt_ckpt_info* info) {
    if (info == nullptr) return fail(GOCKPT_EINVAL, "read_checkpoint_info: info is NULL");
    Meta m;
    const int rc = load_meta(dir, &m);
    if (rc != GOCKPT_OK) return rc;
    to_info(m, info);
    return GOCKPT_OK;
}

int gockpt_read_checkpoint(const char* dir, int64_t n, float* master, float* exp_avg, float* exp_avg_sq,
                           gockpt_ckpt_info* info, int nthreads, gockpt_io_stats* stats) {
    const auto t0 = std::chrono::steady_clock::now();
    Meta m;
    int rc = load_meta(dir, &m);
    if (rc != GOCKPT_OK) return rc;
    if (m.n != n) return fail(GOCKPT_EINVAL, "read_checkpoint: the checkpoint holds " + std::to_string(m.n) +
                                                 " elements, the caller asked for " + std::to_string(n));
    if (n > 0 && (master == nullptr || exp_avg == nullptr || exp_avg_sq == nullptr))
        return fail(GOCKPT_EINVAL, "read_checkpoint: NULL array");
    const Layout L = make_layout(m.n, m.piece);
    const std::string data_path = path_join(dir, "data.bin");
    const int fd = open(data_path.c_str(), O_RDONLY);
    if (fd < 0) return fail(GOCKPT_EFAILED, std::string("read_checkpoint: open data.bin: ") + strerror(errno));
    struct stat st;
    if (fstat(fd, &st) != 0 || static_cast<uint64_t>(st.st_size) < L.total) {
        close(fd);
        return fail(GOCKPT_EFAILED, "read_checkpoint: data.bin is shorter than the checkpoint");
    }
    uint8_t* dst[3] = {reinterpret_cast<uint8_t*>(master), reinterpret_cast<uint8_t*>(exp_avg),
                       reinterpret_cast<uint8_t*>(exp_avg_sq)};
    std::atomic<int64_t> bad{-1};
    std::atomic<int> io_errno{0};  // errno is per thread: keep the reader's
    const bool ok = parallel_pieces(L.pieces.size(), nthreads, [&](size_t k) {
        const Piece& p = L.pieces[k];
        uint8_t* d = dst[p.array] + p.offset;
        if (!pread_all(fd, d, p.bytes, p.array * L.stride + p.offset)) {
            io_errno = errno;
            return false;
        }
        const size_t idx = k - L.first[p.array];
        if (crc32c(d, p.bytes) != m.crc[p.array][idx]) {
            bad = static_cast<int64_t>(k);
            return false;
        }
        return true;
    });
    close(fd);
    if (!ok) {
        if (bad.load() >= 0) {
            const Piece& p = L.pieces[static_cast<size_t>(bad.load())];
            const char* names[3] = {"master", "exp_avg", "exp_avg_sq"};
            return fail(GOCKPT_EFAILED, std::string("read_checkpoint: checksum mismatch in ") + names[p.array] +
                                            " at byte " + std::to_string(p.offset));
        }
        return fail(GOCKPT_EFAILED, std::string("read_checkpoint: reading data.bin: ") +
                                        (io_errno.load() ? strerror(io_errno.load()) : "short read"));
    }
    if (info != nullptr) to_info(m, info);
    if (stats != nullptr) {
        stats->bytes = static_cast<double>(3 * L.array_bytes);
        stats->ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
        stats->pieces = static_cast<int64_t>(L.pieces.size());
    }
    return GOCKPT_OK;
}

int gockpt_read_checkpoint_user(const char* dir, char* buf, size_t capacity, size_t* length) {
    Meta m;
    const int rc = load_meta(dir, &m);
    if (rc != GOCKPT_OK) return rc;
    std::string text;
    if (m.has_user && !read_file(path_join(dir, "user"), &text))
        return fail(GOCKPT_EFAILED, "read_checkpoint_user: user file missing");
    if (length != nullptr) *length = text.size();
    if (buf != nullptr) {
        if (capacity < text.size() + 1) return fail(GOCKPT_ENOMEM, "read_checkpoint_user: buffer too small");
        memcpy(buf, text.data(), text.size());
        buf[text.size()] = '\0';
    }
    return GOCKPT_OK;
}

int gockpt_find_latest_checkpoint(const char* root, char* out, size_t capacity) {
    if (root == nullptr || out == nullptr) return fail(GOCKPT_EINVAL, "find_latest_checkpoint: bad arguments");
    DIR* d = opendir(root);
    if (d == nullptr) return fail(GOCKPT_EFAILED, std::string("find_latest_checkpoint: opendir ") + root);
    std::string best_name;
    int64_t best_t = -1;
    while (const dirent* e = readdir(d)) {
        const std::string name = e->d_name;
        if (name == "." || name == "..") continue;
        const std::string sub = path_join(root, name.c_str());
        struct stat st;
        if (stat(sub.c_str(), &st) != 0 || !S_ISDIR(st.st_mode)) continue;
        std::string text, err;
        Meta m;
        if (!read_file(path_join(sub.c_str(), "meta"), &text) || !parse_meta(text, &m, err)) continue;
        if (m.t > best_t || (m.t == best_t && name > best_name)) {
            best_t = m.t;
            best_name = name;
        }
    }
    closedir(d);
    if (best_t < 0) return fail(GOCKPT_EFAILED, std::string("no complete checkpoint under ") + root);
    const std::string path = path_join(root, best_name.c_str());
    if (capacity < path.size() + 1) return fail(GOCKPT_ENOMEM, "find_latest_checkpoint: buffer too small");
    memcpy(out, path.c_str(), path.size() + 1);
    return GOCKPT_OK;
}

}  // extern "C"
