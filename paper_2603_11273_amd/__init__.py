"""MI355X-native batched Whisper-shaped ASR step behind a duration-aware queue.

Importing the package loads nothing native; `paper_2603_11273_amd.asr`
loads the HIP library and raises if it is missing.
"""
