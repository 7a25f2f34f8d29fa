"""MI355X (gfx950) library for the vocabulary-wide logits path of online
speculative decoding (Liu et al., arXiv:2310.07177).

    osd_verify             speculative-sampling verification (Appendix A.1, Eq. 5)
    osd_verify_noalloc     the same without a workspace (library-held scratch)
    osd_distill_loss_grad  FKL / RKL / JSD[beta] distillation loss and gradient
                           with respect to the draft logits (Section 4.1, Eq. 2-4)
    osd_verify_distill     both of one step in one pass over the row pairs
    osd_verify_distill_rejected  the same, distilling each sequence's first
                           rejected row (Algorithm 1's error index)
    osd_verify_tree        multi-candidate (tree) verification (Medusa-style
                           candidate trees; Section 5)
    osd_sample             proposal sampling y ~ q and mixed sampling
                           y ~ beta p + (1 - beta) q (Algorithm 1; Section 4.1)
    osd_shard_verify_*     verification with the vocabulary split over ranks
                           (stats, mass, draw: one call per phase per rank)

The computation lives in libosd.so (C ABI: include/osd.h); this package is
argument marshalling over it.  Build with ``python -m paper_2310_07177_amd.build``.
"""
from .binding import (OSD_BF16, OSD_F32, OSD_FKL, OSD_JSD, OSD_MAX_K, OSD_RKL, OsdError,  # noqa: F401
                      lib, osd_distill_loss_grad, osd_max_vocab, osd_sample, osd_shard_verify_draw,
                      osd_shard_verify_mass, osd_shard_verify_stats, osd_verify, osd_verify_distill,
                      osd_verify_distill_rejected, osd_verify_noalloc, osd_verify_tree)
