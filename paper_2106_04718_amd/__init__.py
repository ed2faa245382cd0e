"""MI355X-native beam-search decode step (FastSeq, arXiv 2106.04718).

* :func:`beam_cross_attn` -- encoder-decoder attention in which the k beams
  of a source share one de-duplicated K/V copy (Appendix B, Eq. 4).
* :func:`beam_prefix_attn` -- self-attention over a split cache: a prefix
  shared by the beams plus per-beam generated tokens (Appendix A, Eq. 2-3).
* :func:`ngram_block` -- GPU no-repeat-n-gram blocking, in place
  (Section 4.2, Algorithm 1).

Both run hand-written gfx950 HIP kernels behind the C ABI of
``include/fastseq_hip.h`` (``libfastseq_hip.so``).  ``workloads`` holds the
seeded synthetic inputs.  Importing the package loads neither torch nor the
library; the first call does.
"""

_API = ("beam_cross_attn", "beam_cross_attn_workspace_bytes", "beam_prefix_attn",
        "beam_prefix_attn_workspace_bytes", "new_workspace", "ngram_block")

__all__ = list(_API)


def __getattr__(name):
    if name in _API:
        from . import api
        return getattr(api, name)
    raise AttributeError(name)
