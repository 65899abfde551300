"""MI355X-native speculative-verification decode step (WAR, arXiv 2607.17299).

The package holds:
  * ``csrc/``   hand-written HIP kernels for gfx950 and the C-ABI runtime
                (built into ``libwar.so`` next to this file);
  * ``war``     the thin ctypes binding over that C-ABI (argument marshalling only);
  * ``synth``   seeded synthetic inputs (weights, cached context, token streams);
  * ``drafter`` the host-side suffix-match drafter that proposes draft tokens.

Nothing is imported eagerly so that the input generators can be used on a
machine without the built library.
"""

__all__ = ["war", "synth", "drafter", "build"]
