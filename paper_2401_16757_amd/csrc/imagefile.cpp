// imagefile.cpp -- the storage tier: the planned weight image in a file.
//
// Direct block fetch (Sec. 4.2.1): the blocks live in external storage and
// a swap-in reads a block with direct I/O, bypassing the page cache, so the
// block is read once, into memory the next step uses as is.  Here the file
// holds the pinned image of one plan, slab after slab in device layout, each
// slab at a 4 KiB-aligned offset and padded to a multiple of 4 KiB, so one
// O_DIRECT read per slab lands the slab in a pinned staging buffer from
// which one DMA moves it into the arena.
//
// Layout (little-endian):
//   header, kFileAlign-padded:
//     char magic[8] = "SNIMAGE1"; uint32 version = 1; uint32 n_slabs;
//     uint64 image_bytes; uint64 header_bytes;
//     n_slabs x { uint64 image_off, bytes, file_off, fnv1a64(slab bytes) }
//   slab i: `bytes` bytes at file_off (then zeros to the next 4 KiB)
#include <errno.h>
#include <fcntl.h>
#include <string.h>
#include <unistd.h>

#include <string>
#include <vector>

#include "engine.h"

namespace sn {

namespace {

constexpr char kMagic[8] = {'S', 'N', 'I', 'M', 'A', 'G', 'E', '1'};
constexpr uint32_t kVersion = 1;
constexpr int64_t kFixed = 32;          // magic, version, n_slabs, image_bytes, header_bytes
constexpr int64_t kPerSlab = 32;        // image_off, bytes, file_off, checksum

// FNV-1a, 64-bit (offset basis 0xcbf29ce484222325, prime 0x100000001b3)
uint64_t fnv1a64(const uint8_t *p, int64_t n) {
    uint64_t h = 0xcbf29ce484222325ull;
    for (int64_t i = 0; i < n; ++i) {
        h ^= p[i];
        h *= 0x100000001b3ull;
    }
    return h;
}

int64_t header_bytes_for(int n) { return align_up(kFixed + kPerSlab * (int64_t)n, kFileAlign); }

void put64(std::vector<uint8_t> &b, int64_t at, uint64_t v) { memcpy(b.data() + at, &v, 8); }
uint64_t get64(const uint8_t *b, int64_t at) {
    uint64_t v;
    memcpy(&v, b + at, 8);
    return v;
}

bool write_all(int fd, const uint8_t *p, int64_t n, int64_t off) {
    while (n > 0) {
        const ssize_t k = pwrite(fd, p, (size_t)n, (off_t)off);
        if (k < 0 && errno == EINTR) continue;
        if (k <= 0) return false;
        p += k;
        n -= k;
        off += k;
    }
    return true;
}

}  // namespace

int64_t image_file_slab_off(const PlanResult &plan, int i) {
    int64_t off = header_bytes_for((int)plan.slabs.size());
    for (int j = 0; j < i; ++j) off += align_up(plan.slabs[j].bytes, kFileAlign);
    return off;
}

int image_file_write(const std::string &path, const PlanResult &plan, const uint8_t *image,
                     std::string &err) {
    const int n = (int)plan.slabs.size();
    const int64_t hb = header_bytes_for(n);
    std::vector<uint8_t> hdr((size_t)hb, 0);
    memcpy(hdr.data(), kMagic, 8);
    memcpy(hdr.data() + 8, &kVersion, 4);
    const uint32_t nn = (uint32_t)n;
    memcpy(hdr.data() + 12, &nn, 4);
    put64(hdr, 16, (uint64_t)plan.image_bytes);
    put64(hdr, 24, (uint64_t)hb);
    for (int i = 0; i < n; ++i) {
        const Slab &s = plan.slabs[i];
        const int64_t at = kFixed + kPerSlab * i;
        put64(hdr, at, (uint64_t)s.image_off);
        put64(hdr, at + 8, (uint64_t)s.bytes);
        put64(hdr, at + 16, (uint64_t)image_file_slab_off(plan, i));
        put64(hdr, at + 24, fnv1a64(image + s.image_off, s.bytes));
    }
    const int fd = open(path.c_str(), O_WRONLY | O_CREAT | O_TRUNC | O_CLOEXEC, 0644);
    if (fd < 0) {
        err = "image file: cannot create " + path + ": " + strerror(errno);
        return SN_E_INVALID;
    }
    bool ok = write_all(fd, hdr.data(), hb, 0);
    static const uint8_t zeros[kFileAlign] = {};
    for (int i = 0; ok && i < n; ++i) {
        const Slab &s = plan.slabs[i];
        const int64_t off = image_file_slab_off(plan, i);
        ok = write_all(fd, image + s.image_off, s.bytes, off);
        const int64_t pad = align_up(s.bytes, kFileAlign) - s.bytes;
        if (ok && pad) ok = write_all(fd, zeros, pad, off + s.bytes);
    }
    if (ok) ok = fsync(fd) == 0;
    const int e = errno;
    close(fd);
    if (!ok) {
        err = "image file: write to " + path + " failed: " + strerror(e);
        return SN_E_INVALID;
    }
    return SN_OK;
}

int image_file_read(int fd, int64_t off, int64_t bytes, uint8_t *dst, std::string &err) {
    int64_t n = align_up(bytes, kFileAlign);
    while (n > 0) {
        const ssize_t k = pread(fd, dst, (size_t)n, (off_t)off);
        if (k < 0 && errno == EINTR) continue;
        if (k <= 0) {
            err = std::string("image file: read failed: ") + (k < 0 ? strerror(errno) : "end of file");
            return SN_E_INVALID;
        }
        dst += k;
        off += k;
        n -= k;
    }
    return SN_OK;
}

int image_file_open(const std::string &path, const PlanResult &plan, std::vector<int64_t> &file_off,
                    bool &direct, std::string &err) {
    int fd = open(path.c_str(), O_RDONLY | O_DIRECT | O_CLOEXEC);
    direct = fd >= 0;
    if (fd < 0 && errno == EINVAL) fd = open(path.c_str(), O_RDONLY | O_CLOEXEC);   // no O_DIRECT here
    if (fd < 0) {
        err = "image file: cannot open " + path + ": " + strerror(errno);
        return -1;
    }
    const int n = (int)plan.slabs.size();
    const int64_t hb = header_bytes_for(n);
    void *buf = nullptr;
    if (posix_memalign(&buf, (size_t)kFileAlign, (size_t)hb) != 0) {
        close(fd);
        err = "image file: header buffer allocation failed";
        return -1;
    }
    std::string rerr;
    bool ok = image_file_read(fd, 0, hb, (uint8_t *)buf, rerr) == SN_OK;
    const uint8_t *h = (const uint8_t *)buf;
    uint32_t ver = 0, nn = 0;
    if (ok) {
        memcpy(&ver, h + 8, 4);
        memcpy(&nn, h + 12, 4);
        ok = memcmp(h, kMagic, 8) == 0 && ver == kVersion && (int)nn == n &&
             (int64_t)get64(h, 16) == plan.image_bytes && (int64_t)get64(h, 24) == hb;
        if (!ok) rerr = "not an image file of this plan (header)";
    }
    file_off.assign(n, 0);
    for (int i = 0; ok && i < n; ++i) {
        const int64_t at = kFixed + kPerSlab * i;
        const Slab &s = plan.slabs[i];
        file_off[i] = (int64_t)get64(h, at + 16);
        ok = (int64_t)get64(h, at) == s.image_off && (int64_t)get64(h, at + 8) == s.bytes &&
             file_off[i] % kFileAlign == 0 && file_off[i] >= hb;
        if (!ok) rerr = "not an image file of this plan (slab " + std::to_string(i) + ")";
    }
    free(buf);
    if (ok) {
        // the file must hold every slab's padded bytes
        const off_t end = lseek(fd, 0, SEEK_END);
        const int64_t need = n ? file_off[n - 1] + align_up(plan.slabs[n - 1].bytes, kFileAlign) : hb;
        ok = end >= (off_t)need;
        if (!ok) rerr = "image file is truncated";
    }
    if (!ok) {
        close(fd);
        err = "image file " + path + ": " + rerr;
        return -1;
    }
    return fd;
}

}  // namespace sn
