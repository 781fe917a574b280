// kernels_d_list.h -- catalogue of direct (global->LDS copy) GO-Kernels for
// one input type; expanded by the kernels_d_*.hip units.  The staged family
// in kernels_list.h holds the same tiles for GEMMs the direct kernels cannot
// take (K not a multiple of the K tile, unaligned).
#define GDY_TILES_D(L, TA, TB)                                        \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 256, 2, 4, 2),     \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 256, 2, 2, 2),     \
  GDY_KERNEL_DH(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 256, 2, 4, 4),    \
  GDY_KERNEL_DH(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 256, 2, 2, 4),    \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 128, 2, 2, 3),     \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 256, 2, 2, 3),     \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 128, 2, 2, 2),     \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 128, 2, 2, 4)

#define GDY_TILES_D_SMALL(L, TA, TB)                                  \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 128, 2, 2, 3),     \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 128, 2, 2, 2)

// Small tiles with deep rings, for GEMMs whose few workgroups each walk a
// long K: there the time per K tile is the memory latency, and the ring keeps
// up to three tiles in flight where the register-staged kernel of the same
// tile keeps one.  32-row tiles for 16-bit types only (an 8-bit 32-row tile
// is too narrow for the k-major copy layout the kernel also instantiates).
#if GDY_DT16
#define GDY_TILES_D_LAT32(L, TA, TB)                                  \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 32, 256, 1, 4, 3),      \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 32, 128, 1, 4, 4),
#else
#define GDY_TILES_D_LAT32(L, TA, TB)
#endif
#define GDY_TILES_D_LAT(L, TA, TB)                                    \
  GDY_TILES_D_LAT32(L, TA, TB)                                        \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 256, 1, 4, 3),      \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 128, 2, 2, 4),      \
  GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 64, 2, 2, 4)

// 16 waves of 64x64 (4 per SIMD): 16-bit types only (fp8 fragments are
// twice as wide and would not fit in 128 registers).
#if GDY_DT16
#define GDY_TILES_D_WIDE(L, TA, TB) GDY_KERNEL_D(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 256, 4, 4, 2),
#else
#define GDY_TILES_D_WIDE(L, TA, TB)
#endif

static const ::gdy::KernelDesc kTableD[] = {
    GDY_TILES_D_WIDE("nn", 0, 0)
    GDY_TILES_D_WIDE("nt", 0, 1)
    GDY_TILES_D("nn", 0, 0),
    GDY_TILES_D("nt", 0, 1),
    GDY_TILES_D_SMALL("tn", 1, 0),
    GDY_TILES_D_SMALL("tt", 1, 1),
    GDY_TILES_D_LAT("nn", 0, 0),
    GDY_TILES_D_LAT("nt", 0, 1),
    GDY_KERNEL_D(GDY_DT, GDY_DTNAME, 1, 0, "tn", 64, 64, 2, 2, 4),
    GDY_KERNEL_D(GDY_DT, GDY_DTNAME, 1, 1, "tt", 64, 64, 2, 2, 4),
};
