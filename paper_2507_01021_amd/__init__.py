"""MI355X-native batched Whisper inference over multiplexed speech segments.

The compute path is the C-ABI library built from ``csrc/`` (hand-written HIP
for gfx950); ``binding`` marshals arguments to it and ``synth`` draws the
seeded synthetic inputs. Importing the package loads nothing native; call
``binding.load()`` (or use ``binding.Context``) to load the library.
"""
__all__ = ["synth", "binding"]
