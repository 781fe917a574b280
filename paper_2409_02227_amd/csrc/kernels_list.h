// kernels_list.h -- the GO-Kernel catalogue: macro tiles x layouts for one
// input type.  Expanded once per type by the kernels_*.hip units, which
// define GDY_DT and GDY_DTNAME before including it.
//
// Tiles span the axes the tuner chooses from: large tiles (more LDS reuse,
// fewer workgroups) down to 16-row tiles for skinny GEMMs; 4 or 8 waves.
#define GDY_TILES(L, TA, TB)                                   \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 256, 2, 4, 32), \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 128, 2, 2, 32), \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 256, 2, 2, 32), \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 128, 2, 2, 32), \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 256, 1, 4, 32),  \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 128, 1, 4, 32),  \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 64, 2, 2, 32),   \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 32, 256, 1, 4, 32),  \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 32, 128, 1, 4, 32),  \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 16, 256, 1, 4, 16),  \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 16, 128, 1, 4, 16),  \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 16, 64, 1, 4, 16)

// Transposed-A layouts carry a smaller set (they are off the timed path).
#define GDY_TILES_SMALL(L, TA, TB)                             \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 256, 128, 2, 2, 32), \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 128, 128, 2, 2, 32), \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 64, 64, 2, 2, 32),   \
  GDY_KERNEL(GDY_DT, GDY_DTNAME, TA, TB, L, 16, 64, 1, 4, 16)

static const ::gdy::KernelDesc kTable[] = {
    GDY_TILES("nn", 0, 0),
    GDY_TILES("nt", 0, 1),
    GDY_TILES_SMALL("tn", 1, 0),
    GDY_TILES_SMALL("tt", 1, 1),
};
