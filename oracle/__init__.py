"""CPU oracle of one MAP-Elites generation -- test infrastructure only."""
